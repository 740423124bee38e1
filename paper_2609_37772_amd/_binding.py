"""ctypes binding of libuad.so: argument marshalling only.

Every function has the name of the C entry point it calls (see include/uad.h)
and does nothing but check/convert arguments and forward them; all device
work runs in the library's HIP kernels.  There is no fallback: if libuad.so is
missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Tuple

import numpy as np
import torch  # loaded first on purpose: libuad then binds to PyTorch's HIP runtime

__all__ = [
    "LIB_PATH", "EXPORTED_SYMBOLS", "UadError", "load_library", "library_loaded",
    "uad_create", "uad_destroy", "uad_last_error", "uad_set_stream", "uad_load_weights",
    "uad_set_prefix_kv", "uad_denoise_step", "uad_denoise_step_static", "uad_denoise_schedule",
    "uad_denoise_budgets", "uad_denoise_release", "uad_build_schedule", "uad_aal", "uad_synchronize", "uad_tick_rate_hz",
    "uad_debug_velocity_field", "uad_profile_enable", "uad_profile_read", "UAD_DTYPE_F32", "UAD_DTYPE_BF16", "STATUS_NAMES",
    "UAD_RELEASE_UAER", "UAD_RELEASE_TR", "UAD_FLAG_ADARMS",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libuad.so")
UAD_DTYPE_F32, UAD_DTYPE_BF16 = 0, 1
UAD_RELEASE_UAER, UAD_RELEASE_TR = 0, 1
UAD_FLAG_ADARMS = 1
STATUS_NAMES = {0: "UAD_OK", 1: "UAD_E_INVALID", 2: "UAD_E_SHAPE", 3: "UAD_E_STATE", 4: "UAD_E_MISSING",
                5: "UAD_E_HIP", 6: "UAD_E_OOM", 7: "UAD_E_UNSUPPORTED", 8: "UAD_E_RANGE"}
EXPORTED_SYMBOLS = [
    "uad_create", "uad_destroy", "uad_last_error", "uad_set_stream", "uad_load_weights",
    "uad_set_prefix_kv", "uad_denoise_step", "uad_denoise_step_static", "uad_denoise_schedule", "uad_denoise_budgets",
    "uad_denoise_release",
    "uad_build_schedule", "uad_aal", "uad_synchronize", "uad_tick_rate_hz", "uad_debug_velocity_field",
    "uad_profile_enable", "uad_profile_read",
]


class UadError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class uad_model_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("action_dim", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_chunk", ctypes.c_int32),
                ("max_prefix", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("flags", ctypes.c_int32)]


class uad_tensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("data", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("ndim", ctypes.c_int32), ("shape", ctypes.c_int64 * 4), ("on_device", ctypes.c_int32)]


_lib: Optional[ctypes.CDLL] = None


def load_library() -> ctypes.CDLL:
    """Load libuad.so (built by ``python -m paper_2609_37772_amd.build``); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_37772_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "uad_create": ([ctypes.POINTER(uad_model_config), I32, P, ctypes.POINTER(P)], I32),
        "uad_destroy": ([P], None),
        "uad_last_error": ([P], ctypes.c_char_p),
        "uad_set_stream": ([P, P], I32),
        "uad_load_weights": ([P, ctypes.POINTER(uad_tensor), I32], I32),
        "uad_set_prefix_kv": ([P, P, P, I32, I32, I32, I32], I32),
        "uad_denoise_step": ([P, P, P, P, P, P, I32, I32], I32),
        "uad_denoise_step_static": ([P, P, P, P, P, P, I32, I32], I32),
        "uad_denoise_schedule": ([P, P, P, P, P, I32, I32, I32, P, P, P], I32),
        "uad_denoise_budgets": ([P, P, P, I32, I32, P, P, P], I32),
        "uad_denoise_release": ([P, P, I32, I32, I32, I32, I32, I32, I32, P, P, P, P, P, P], I32),
        "uad_build_schedule": ([P, I32, I32, I32, P, P, P, P], I32),
        "uad_aal": ([P, I32, ctypes.c_double, P], I32),
        "uad_synchronize": ([P], I32),
        "uad_tick_rate_hz": ([P, P], I32),
        "uad_debug_velocity_field": ([P, I32, F32, F32], I32),
        "uad_profile_enable": ([P, I32], I32),
        "uad_profile_read": ([P, I32, ctypes.c_char_p, I32, P, P], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def library_loaded() -> bool:
    return _lib is not None


def _check(ctx, st: int, what: str):
    if st != 0:
        msg = load_library().uad_last_error(ctx)
        raise UadError(st, f"{what}: {msg.decode() if msg else ''}")


def _dev_ptr(t: Optional[torch.Tensor], dtype: torch.dtype, shape: Tuple[int, ...], name: str) -> Optional[int]:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


# ----------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ----------------------------------------------------------------------------
def uad_create(shape, max_batch: int, max_chunk: int, max_prefix: int, device: int = 0,
               stream: Optional[torch.cuda.Stream] = None) -> int:
    """Create a context for a model shape (fields as ``uad_workloads.ModelShape``); returns a handle."""
    lib = load_library()
    flags = UAD_FLAG_ADARMS if getattr(shape, "conditioning", "input") == "adarms" else 0
    cfg = uad_model_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                           shape.d_ff, shape.action_dim, max_batch, max_chunk, max_prefix,
                           float(shape.rms_eps), flags)
    if stream is None:
        stream = torch.cuda.current_stream(device)
    out = ctypes.c_void_p()
    st = lib.uad_create(ctypes.byref(cfg), device, ctypes.c_void_p(stream.cuda_stream), ctypes.byref(out))
    _check(None, st, "uad_create")
    return out.value


def uad_destroy(ctx: int) -> None:
    load_library().uad_destroy(ctx)


def uad_last_error(ctx: Optional[int]) -> str:
    m = load_library().uad_last_error(ctx)
    return m.decode() if m else ""


def uad_set_stream(ctx: int, stream: Optional[torch.cuda.Stream]) -> None:
    _check(ctx, load_library().uad_set_stream(ctx, None if stream is None else stream.cuda_stream), "uad_set_stream")


def _raw(name: str, a):
    """(pointer, uad dtype, on_device, shape, keep-alive) of an fp32 / bf16 array or tensor."""
    if isinstance(a, torch.Tensor):
        keep = a.contiguous()
        if keep.dtype == torch.float32:
            dt = UAD_DTYPE_F32
        elif keep.dtype == torch.bfloat16:
            dt = UAD_DTYPE_BF16
        else:
            raise ValueError(f"{name}: dtype {keep.dtype} not supported")
        return keep.data_ptr(), dt, int(keep.is_cuda), tuple(keep.shape), keep
    keep = np.ascontiguousarray(a)
    if keep.dtype == np.float32:
        dt = UAD_DTYPE_F32
    elif keep.dtype == np.uint16:
        dt = UAD_DTYPE_BF16
    else:
        raise ValueError(f"{name}: dtype {keep.dtype} not supported (float32 or bf16 bits as uint16)")
    return keep.ctypes.data, dt, 0, tuple(keep.shape), keep


def _as_tensor_struct(name: str, a) -> Tuple[uad_tensor, object]:
    if isinstance(a, torch.Tensor):
        keep = a.contiguous()
        if keep.dtype == torch.float32:
            dt = UAD_DTYPE_F32
        elif keep.dtype == torch.bfloat16:
            dt = UAD_DTYPE_BF16
        else:
            raise ValueError(f"{name}: dtype {keep.dtype} not supported")
        ptr, on_dev, shape = keep.data_ptr(), int(keep.is_cuda), tuple(keep.shape)
    else:
        keep = np.ascontiguousarray(a)
        if keep.dtype == np.float32:
            dt = UAD_DTYPE_F32
        elif keep.dtype == np.uint16:
            dt = UAD_DTYPE_BF16
        else:
            raise ValueError(f"{name}: dtype {keep.dtype} not supported (float32 or bf16 bits as uint16)")
        ptr, on_dev, shape = keep.ctypes.data, 0, keep.shape
    if len(shape) > 4:
        raise ValueError(f"{name}: more than 4 dims")
    s = uad_tensor(name.encode(), ptr, dt, len(shape), (ctypes.c_int64 * 4)(*(list(shape) + [0] * (4 - len(shape)))),
                   on_dev)
    return s, keep


def uad_load_weights(ctx: int, weights: Dict[str, object]) -> None:
    """Copy named weights (numpy fp32 / uint16 bf16 bits, or torch fp32 / bf16) into the library."""
    structs, keep = [], []
    for k, v in weights.items():
        s, kp = _as_tensor_struct(k, v)
        structs.append(s)
        keep.append(kp)
    arr = (uad_tensor * len(structs))(*structs)
    _check(ctx, load_library().uad_load_weights(ctx, arr, len(structs)), "uad_load_weights")


def uad_set_prefix_kv(ctx: int, k, v, batch: int, prefix_len: int) -> None:
    """Copy prefix K and V ([L][batch][P][Hkv][hd], fp32 / bf16) into the library's K/V store."""
    pk, dk, ok, shk, kk = _raw("prefix_k", k)
    pv, dv, ov, shv, kv = _raw("prefix_v", v)
    if dk != dv or ok != ov or shk != shv:
        raise ValueError("prefix k and v must share dtype, location and shape")
    if len(shk) != 5 or shk[1] != batch or shk[2] != prefix_len:
        raise ValueError(f"prefix k/v must be [L][{batch}][{prefix_len}][Hkv][hd], got {shk}")
    st = load_library().uad_set_prefix_kv(ctx, pk, pv, dk, batch, prefix_len, ok)
    _check(ctx, st, "uad_set_prefix_kv")


def uad_denoise_step(ctx: int, x: torch.Tensor, t: torch.Tensor, dt: torch.Tensor, mask: torch.Tensor,
                     v_out: Optional[torch.Tensor] = None) -> None:
    """One joint step on device tensors: x [B][H][Da] fp32 in/out, t/dt [B][H] fp32, mask [B][H] uint8."""
    B, H, Da = x.shape
    p = [_dev_ptr(x, torch.float32, (B, H, Da), "x"), _dev_ptr(t, torch.float32, (B, H), "t"),
         _dev_ptr(dt, torch.float32, (B, H), "dt"), _dev_ptr(mask, torch.uint8, (B, H), "mask"),
         _dev_ptr(v_out, torch.float32, (B, H, Da), "v_out")]
    _check(ctx, load_library().uad_denoise_step(ctx, *p, B, H), "uad_denoise_step")


def uad_denoise_step_static(ctx: int, x: torch.Tensor, t: torch.Tensor, dt: torch.Tensor, mask: torch.Tensor,
                            v_out: Optional[torch.Tensor] = None) -> None:
    """uad_denoise_step without any allocation (split-KV scratch in a static device array)."""
    B, H, Da = x.shape
    p = [_dev_ptr(x, torch.float32, (B, H, Da), "x"), _dev_ptr(t, torch.float32, (B, H), "t"),
         _dev_ptr(dt, torch.float32, (B, H), "dt"), _dev_ptr(mask, torch.uint8, (B, H), "mask"),
         _dev_ptr(v_out, torch.float32, (B, H, Da), "v_out")]
    _check(ctx, load_library().uad_denoise_step_static(ctx, *p, B, H), "uad_denoise_step_static")


def uad_denoise_schedule(ctx: int, x: torch.Tensor, t_sched: torch.Tensor, dt_sched: torch.Tensor,
                         mask_sched: torch.Tensor, released: Optional[torch.Tensor] = None,
                         release_step: Optional[torch.Tensor] = None,
                         step_ticks: Optional[torch.Tensor] = None) -> None:
    """A whole schedule: tables [n_steps][B][H] on device; step_ticks: pinned host uint64 [n_steps+1]."""
    B, H, Da = x.shape
    n = t_sched.shape[0]
    p = [_dev_ptr(x, torch.float32, (B, H, Da), "x"), _dev_ptr(t_sched, torch.float32, (n, B, H), "t_sched"),
         _dev_ptr(dt_sched, torch.float32, (n, B, H), "dt_sched"),
         _dev_ptr(mask_sched, torch.uint8, (n, B, H), "mask_sched")]
    rel = _dev_ptr(released, torch.float32, (B, H, Da), "released")
    rst = _dev_ptr(release_step, torch.int32, (B, H), "release_step")
    tk = None
    if step_ticks is not None:
        if step_ticks.is_cuda or not step_ticks.is_pinned() or step_ticks.dtype != torch.uint64 \
                or tuple(step_ticks.shape) != (n + 1,):
            raise ValueError("step_ticks must be a pinned host uint64 tensor of n_steps+1 entries")
        tk = step_ticks.data_ptr()
    st = load_library().uad_denoise_schedule(ctx, *p, n, B, H, rel, rst, tk)
    _check(ctx, st, "uad_denoise_schedule")


def uad_denoise_budgets(ctx: int, x: torch.Tensor, budgets: np.ndarray, released: Optional[torch.Tensor] = None,
                        release_step: Optional[torch.Tensor] = None,
                        step_ticks: Optional[torch.Tensor] = None) -> None:
    """A schedule from host int budgets [B][H] (tables built by the library, finished environments skipped)."""
    B, H, Da = x.shape
    bud = np.ascontiguousarray(budgets, np.int32)
    if bud.shape != (B, H):
        raise ValueError(f"budgets must be [{B}][{H}], got {bud.shape}")
    px = _dev_ptr(x, torch.float32, (B, H, Da), "x")
    rel = _dev_ptr(released, torch.float32, (B, H, Da), "released")
    rst = _dev_ptr(release_step, torch.int32, (B, H), "release_step")
    tk = None
    if step_ticks is not None:
        n = int(bud.max())
        if step_ticks.is_cuda or not step_ticks.is_pinned() or step_ticks.dtype != torch.uint64 \
                or tuple(step_ticks.shape) != (n + 1,):
            raise ValueError("step_ticks must be a pinned host uint64 tensor of max(budgets)+1 entries")
        tk = step_ticks.data_ptr()
    st = load_library().uad_denoise_budgets(ctx, px, bud.ctypes.data, B, H, rel, rst, tk)
    _check(ctx, st, "uad_denoise_budgets")


def uad_denoise_release(ctx: int, x: torch.Tensor, U: int, K: int, Nstar: int, S: int, mode: int,
                        urgent: torch.Tensor, executed: Optional[torch.Tensor] = None,
                        gac_mask: Optional[torch.Tensor] = None, urgent_host: Optional[torch.Tensor] = None,
                        release_event: Optional["torch.cuda.Event"] = None,
                        step_ticks: Optional[torch.Tensor] = None) -> None:
    """Urgency-aware release of a chunk per environment (UAER or TR, GAC with ``executed``).

    x [B][H][Da] device fp32 in/out; urgent [B][U][Da] device; executed [B][S][Da] device;
    gac_mask [Da] device uint8; urgent_host [B][U][Da] pinned host fp32; release_event a
    torch.cuda.Event recorded when the urgent actions are final; step_ticks pinned uint64 [N*+1].
    """
    B, H, Da = x.shape
    px = _dev_ptr(x, torch.float32, (B, H, Da), "x")
    pu = _dev_ptr(urgent, torch.float32, (B, U, Da), "urgent")
    pe = _dev_ptr(executed, torch.float32, (B, S, Da), "executed")
    pm = _dev_ptr(gac_mask, torch.uint8, (Da,), "gac_mask")
    ph = None
    if urgent_host is not None:
        if urgent_host.is_cuda or not urgent_host.is_pinned() or urgent_host.dtype != torch.float32 \
                or tuple(urgent_host.shape) != (B, U, Da):
            raise ValueError("urgent_host must be a pinned host fp32 tensor [B][U][Da]")
        ph = urgent_host.data_ptr()
    ev = None
    if release_event is not None:
        release_event.record()  # materialise the event before handing its handle over
        ev = release_event.cuda_event
    tk = None
    if step_ticks is not None:
        if step_ticks.is_cuda or not step_ticks.is_pinned() or step_ticks.dtype != torch.uint64 \
                or tuple(step_ticks.shape) != (Nstar + 1,):
            raise ValueError("step_ticks must be a pinned host uint64 tensor of N*+1 entries")
        tk = step_ticks.data_ptr()
    st = load_library().uad_denoise_release(ctx, px, B, H, U, K, Nstar, S, mode, pu, pe, pm, ph, ev, tk)
    _check(ctx, st, "uad_denoise_release")


def uad_build_schedule(budgets: np.ndarray, max_steps: int = 64):
    """Host schedule tables from int budgets [B][H]: (n_steps, t, dt, mask) numpy arrays [n][B][H]."""
    bud = np.ascontiguousarray(budgets, np.int32)
    B, H = bud.shape
    t = np.zeros((max_steps, B, H), np.float32)
    dt = np.zeros_like(t)
    mask = np.zeros((max_steps, B, H), np.uint8)
    n = ctypes.c_int32(0)
    st = load_library().uad_build_schedule(bud.ctypes.data, B, H, max_steps, ctypes.addressof(n),
                                           t.ctypes.data, dt.ctypes.data, mask.ctypes.data)
    if st != 0:
        raise UadError(st, "uad_build_schedule: invalid budgets or sizes")
    k = n.value
    return k, t[:k].copy(), dt[:k].copy(), mask[:k].copy()


def uad_aal(release, t_act: float) -> float:
    r = np.ascontiguousarray(release, np.float64)
    out = ctypes.c_double(0)
    st = load_library().uad_aal(r.ctypes.data, len(r), float(t_act), ctypes.addressof(out))
    if st != 0:
        raise UadError(st, "uad_aal: invalid arguments")
    return out.value


def uad_synchronize(ctx: int) -> None:
    _check(ctx, load_library().uad_synchronize(ctx), "uad_synchronize")


def uad_tick_rate_hz(ctx: int) -> float:
    out = ctypes.c_double(0)
    _check(ctx, load_library().uad_tick_rate_hz(ctx, ctypes.addressof(out)), "uad_tick_rate_hz")
    return out.value


def uad_debug_velocity_field(ctx: int, enable: bool, alpha: float = 0.0, beta: float = 0.0) -> None:
    _check(ctx, load_library().uad_debug_velocity_field(ctx, int(enable), float(alpha), float(beta)),
           "uad_debug_velocity_field")


def uad_profile_enable(ctx: int, enable: bool) -> None:
    _check(ctx, load_library().uad_profile_enable(ctx, int(enable)), "uad_profile_enable")


def uad_profile_read(ctx: int) -> Dict[str, Tuple[float, int]]:
    """{kernel class: (total event-measured ms, launches)} since profiling was enabled."""
    lib = load_library()
    out = {}
    i = 0
    while True:
        name = ctypes.create_string_buffer(64)
        ms = ctypes.c_double(0)
        n = ctypes.c_int64(0)
        st = lib.uad_profile_read(ctx, i, name, 64, ctypes.addressof(ms), ctypes.addressof(n))
        if st != 0:
            break
        out[name.value.decode()] = (ms.value, n.value)
        i += 1
    return out
