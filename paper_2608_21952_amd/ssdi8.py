"""Python binding of libssdi8 (include/ssdi8.h): argument marshalling only.

Every step of the SSD path runs in the library's HIP kernels; this module checks tensor
placement/dtype/shape, allocates outputs and the workspace with PyTorch (device memory and
streams are PyTorch's job here), and forwards raw device pointers and the current HIP stream.
There is no fallback: if the shared library is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Iterable, Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libssdi8.so")

OK, ERR_NULL, ERR_SHAPE, ERR_UNSUPPORTED, ERR_ALIGN, ERR_WORKSPACE, ERR_HIP, ERR_ARG = range(8)
F32, F16 = 0, 1
GRAN = {"tensor": 0, "group": 1, "channel": 2, "token": 3}
P_DIM, N_DIM, CHUNK = 64, 128, 256


class SSDi8Error(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("batch", "seqlen", "nheads", "headdim", "ngroups", "dstate", "chunk")]


_P = ctypes.c_void_p
_I = ctypes.c_int


class ScanArgs(ctypes.Structure):
    _fields_ = [
        ("x", _P), ("x_dtype", _I), ("dt", _P), ("dt_softplus", _I), ("A", _P),
        ("Bq", _P), ("Cq", _P), ("B_scale", _P), ("C_scale", _P), ("c_per_token", _I),
        ("D", _P), ("corr", _P), ("xs_scale", _P), ("xs_per_head", _I), ("state_scale", _P),
        ("cb_scale", _P), ("decay_shift", _I), ("shift_round", _I), ("init_state_q", _P),
        ("y", _P), ("y_dtype", _I), ("final_state_q", _P), ("final_state", _P),
        ("xs_q", _P), ("state_i32", _P), ("state_q", _P), ("decay_q", _P), ("state_in_q", _P),
        ("cb_i32", _P), ("cb_q", _P), ("scan1_i32", _P),
        ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
        ("stage_events", _P), ("path", _I),
        ("B", _P), ("C", _P), ("bc_dtype", _I), ("dt_post", _P), ("hand_off_timeouts", _P),
    ]


class DecodeArgs(ctypes.Structure):
    _fields_ = [
        ("x", _P), ("x_dtype", _I), ("dt", _P), ("dt_softplus", _I), ("A", _P),
        ("Bq", _P), ("Cq", _P), ("B_scale", _P), ("C_scale", _P), ("c_per_token", _I),
        ("D", _P), ("corr", _P), ("xs_scale", _P), ("xs_per_head", _I), ("state_scale", _P),
        ("cb_scale", _P), ("decay_shift", _I), ("shift_round", _I), ("state_q", _P),
        ("y", _P), ("y_dtype", _I), ("state", _P),
    ]


class Fp16Args(ctypes.Structure):
    _fields_ = [
        ("x", _P), ("x_dtype", _I), ("dt", _P), ("dt_softplus", _I), ("A", _P),
        ("B", _P), ("C", _P), ("bc_dtype", _I), ("D", _P), ("init_state", _P),
        ("y", _P), ("y_dtype", _I), ("final_state", _P),
        ("workspace", _P), ("workspace_bytes", ctypes.c_size_t), ("stage_events", _P),
    ]


PATHS = {"auto": 0, "separate": 1, "single": 2}


class CalibArgs(ctypes.Structure):
    _fields_ = [
        ("x", _P), ("x_dtype", _I), ("dt", _P), ("dt_softplus", _I), ("A", _P),
        ("B", _P), ("C", _P), ("bc_dtype", _I), ("D", _P), ("xs_per_head", _I),
        ("eta", ctypes.c_float), ("decay_shift", _I), ("shift_round", _I),
        ("B_scale", _P), ("C_scale", _P), ("xs_scale", _P), ("state_scale", _P),
        ("cb_scale", _P), ("corr", _P),
        ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} not found: build it with "
                          "`python -m paper_2608_21952_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    i64 = ctypes.c_int64
    L.ssdi8_quantize_act.argtypes = [_P, _I, i64, i64, i64, i64, _I, _P, _I, _P, _P]
    L.ssdi8_quantize_act.restype = _I
    L.ssdi8_state_pass.argtypes = [_P, _P, _I, _I, _P, _P, _P, _P, _P, i64, i64, i64, i64, i64,
                                   _P]
    L.ssdi8_state_pass.restype = _I
    L.ssdi8_ssd_workspace_size.argtypes = [ctypes.POINTER(Dims)]
    L.ssdi8_ssd_workspace_size.restype = ctypes.c_size_t
    L.ssdi8_ssd_chunk_scan.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(ScanArgs), _P]
    L.ssdi8_ssd_chunk_scan.restype = _I
    L.ssdi8_ssd_chunk_scan_noalloc.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(ScanArgs),
                                               _P]
    L.ssdi8_ssd_chunk_scan_noalloc.restype = _I
    L.ssdi8_uses_single_pass.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(ScanArgs)]
    L.ssdi8_uses_single_pass.restype = _I
    L.ssdi8_decode_step.argtypes = [i64, i64, i64, i64, i64, ctypes.POINTER(DecodeArgs), _P]
    L.ssdi8_decode_step.restype = _I
    L.ssdi8_fp16_workspace_size.argtypes = [ctypes.POINTER(Dims)]
    L.ssdi8_fp16_workspace_size.restype = ctypes.c_size_t
    L.ssdi8_ssd_chunk_scan_fp16.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(Fp16Args), _P]
    L.ssdi8_ssd_chunk_scan_fp16.restype = _I
    L.ssdi8_calibrate_workspace_size.argtypes = [ctypes.POINTER(Dims)]
    L.ssdi8_calibrate_workspace_size.restype = ctypes.c_size_t
    L.ssdi8_calibrate.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(CalibArgs), _P]
    L.ssdi8_calibrate.restype = _I
    L.ssdi8_mfma_probe.argtypes = [_I, ctypes.c_int64, ctypes.c_int64, _P,
                                   ctypes.POINTER(ctypes.c_int64), _P]
    L.ssdi8_mfma_probe.restype = _I
    L.ssdi8_status_string.argtypes = [_I]
    L.ssdi8_status_string.restype = ctypes.c_char_p
    L.ssdi8_version.argtypes = []
    L.ssdi8_version.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().ssdi8_status_string(int(status)).decode()


def version() -> str:
    return lib().ssdi8_version().decode()


def _check(status: int, where: str) -> None:
    if status != OK:
        raise SSDi8Error(status, where)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _need(t: torch.Tensor, name: str, dtype=None, shape=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _fdt(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return F16
    if t.dtype == torch.float32:
        return F32
    raise ValueError(f"unsupported dtype {t.dtype}")


# ------------------------------------------------------------------------------------- calls
def quantize_act(src: torch.Tensor, gran: str = "group", scale: Optional[torch.Tensor] = None,
                 out: Optional[torch.Tensor] = None, stream=None
                 ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Eq. 1 quantization of a (b, l, k, m) activation.  With `scale` the steps are static;
    without, they are computed on the device (absmax/127 per granule) and returned."""
    _need(src, "src")
    if src.dim() != 4:
        raise ValueError("src must be (b, l, k, m)")
    b, l, k, m = src.shape
    nscale = {"tensor": 1, "group": k, "channel": k * m, "token": b * l * k}[gran]
    dynamic = scale is None
    if dynamic:
        scale = torch.empty(nscale, dtype=torch.float32, device=src.device)
    _need(scale, "scale", torch.float32)
    if scale.numel() != nscale:
        raise ValueError(f"scale must have {nscale} elements for gran={gran}")
    if out is None:
        out = torch.empty(src.shape, dtype=torch.int8, device=src.device)
    _need(out, "out", torch.int8, src.shape)
    st = lib().ssdi8_quantize_act(_ptr(src), _fdt(src), b, l, k, m, GRAN[gran], _ptr(scale),
                                  int(dynamic), _ptr(out), _stream(stream))
    _check(st, "ssdi8_quantize_act")
    return out, scale


def state_pass(state_q: torch.Tensor, decay_q: torch.Tensor, shift: int = 7,
               shift_round: bool = True, init_q: Optional[torch.Tensor] = None,
               state_scale: Optional[torch.Tensor] = None, stream=None
               ) -> Dict[str, torch.Tensor]:
    """Eq. 9 INT8 state passing.  state_q (b, c, h, p, n) int8, decay_q (b, h, c) int16.
    Returns state_in_q (b, c, h, p, n), final_q (b, h, p, n) and, with state_scale (h, p),
    final_state fp32."""
    _need(state_q, "state_q", torch.int8)
    b, c, h, p, n = state_q.shape
    _need(decay_q, "decay_q", torch.int16, (b, h, c))
    if init_q is not None:
        _need(init_q, "init_q", torch.int8, (b, h, p, n))
    dev = state_q.device
    pin = torch.empty_like(state_q)
    fin = torch.empty((b, h, p, n), dtype=torch.int8, device=dev)
    fst = None
    if state_scale is not None:
        _need(state_scale, "state_scale", torch.float32, (h, p))
        fst = torch.empty((b, h, p, n), dtype=torch.float32, device=dev)
    st = lib().ssdi8_state_pass(_ptr(state_q), _ptr(decay_q), shift, int(shift_round),
                                _ptr(init_q), _ptr(pin), _ptr(fin), _ptr(fst), _ptr(state_scale),
                                b, c, h, p, n, _stream(stream))
    _check(st, "ssdi8_state_pass")
    out = {"state_in_q": pin, "final_q": fin}
    if fst is not None:
        out["final_state"] = fst
    return out


def dims(batch: int, seqlen: int, nheads: int, ngroups: int, headdim: int = P_DIM,
         dstate: int = N_DIM, chunk: int = CHUNK) -> Dims:
    return Dims(batch, seqlen, nheads, headdim, ngroups, dstate, chunk)


def workspace_size(d: Dims) -> int:
    return int(lib().ssdi8_ssd_workspace_size(ctypes.byref(d)))


TAPS = {  # name -> (dtype, shape builder(B, L, H, P, G, N, Q, c))
    "xs_q": (torch.int8, lambda B, L, H, P, G, N, Q, c: (B, L, H, P)),
    "dt_post": (torch.float32, lambda B, L, H, P, G, N, Q, c: (B, L, H)),
    "state_i32": (torch.int32, lambda B, L, H, P, G, N, Q, c: (B, c, H, P, N)),
    "state_q": (torch.int8, lambda B, L, H, P, G, N, Q, c: (B, c, H, P, N)),
    "decay_q": (torch.int16, lambda B, L, H, P, G, N, Q, c: (B, H, c)),
    "state_in_q": (torch.int8, lambda B, L, H, P, G, N, Q, c: (B, c, H, P, N)),
    "cb_i32": (torch.int32, lambda B, L, H, P, G, N, Q, c: (B, c, G, Q, Q)),
    "cb_q": (torch.int8, lambda B, L, H, P, G, N, Q, c: (B, c, G, Q, Q)),
    "scan1_i32": (torch.int32, lambda B, L, H, P, G, N, Q, c: (B, L, H, P)),
}


def ssd_chunk_scan(x: torch.Tensor, dt: torch.Tensor, A: torch.Tensor,
                   Bq: Optional[torch.Tensor], Cq: Optional[torch.Tensor],
                   B_scale: torch.Tensor, C_scale: torch.Tensor,
                   xs_scale: torch.Tensor, state_scale: torch.Tensor, cb_scale: torch.Tensor, *,
                   D: Optional[torch.Tensor] = None, corr: Optional[torch.Tensor] = None,
                   dt_softplus: bool = True, chunk: int = CHUNK, decay_shift: int = 7,
                   shift_round: bool = True, init_state_q: Optional[torch.Tensor] = None,
                   y_dtype: Optional[torch.dtype] = None, final_state: bool = True,
                   taps: Iterable[str] = (), workspace: Optional[torch.Tensor] = None,
                   y: Optional[torch.Tensor] = None, stage_events=None,
                   path: str = "auto", B: Optional[torch.Tensor] = None,
                   C: Optional[torch.Tensor] = None, stream=None,
                   hand_off_timeouts: Optional[torch.Tensor] = None,
                   _noalloc: bool = False) -> Dict[str, torch.Tensor]:
    """One SSDi8 SSD layer (ssdi8_ssd_chunk_scan).  Shapes: x (B,L,H,P), dt (B,L,H), A (H),
    Bq/Cq (B,L,G,N) int8 -- or Bq = Cq = None and B, C (B,L,G,N) fp16/fp32 unquantized, then
    quantized with the static B_scale, C_scale inside ChunkBMM --, B_scale (G), C_scale (G) or
    (B,L,G) for per-token C steps,
    xs_scale (H,P) or (H), state_scale (H,P), cb_scale (G), D (H), corr (H,P).
    Returns y, final_state_q, final_state and the requested taps (zero-initialised tensors,
    so entries a stage does not write, such as C.B^T above the diagonal, read as 0).
    path: "auto", "separate" (ChunkState, StatePassing, ChunkScan kernels) or "single" (the
    single-pass kernel whenever x is fp16 and no stage tap other than state_in_q is requested).
    hand_off_timeouts: an int32 device tensor of one element, or None; receives the number of
    single-pass waits that ran out (non-zero: the results of the call are not to be used)."""
    _need(x, "x")
    Bsrc, Csrc = (Bq, Cq) if Bq is not None else (B, C)
    B, L, H, P = x.shape
    if Bq is not None:
        _need(Bq, "Bq", torch.int8)
        if C is not None:
            raise ValueError("pass either Bq, Cq or B, C")
    elif Bsrc is None or Csrc is None:
        raise ValueError("Bq, Cq or B, C are required")
    G, N = Bsrc.shape[2], Bsrc.shape[3]
    _need(Bsrc, "B", Bsrc.dtype, (B, L, G, N))
    _need(Csrc, "C", Bsrc.dtype, (B, L, G, N))
    _need(dt, "dt", torch.float32, (B, L, H))
    _need(A, "A", torch.float32, (H,))
    _need(B_scale, "B_scale", torch.float32, (G,))
    c_per_token = C_scale.dim() == 3
    _need(C_scale, "C_scale", torch.float32, (B, L, G) if c_per_token else (G,))
    xs_per_head = xs_scale.dim() == 1
    _need(xs_scale, "xs_scale", torch.float32, (H,) if xs_per_head else (H, P))
    _need(state_scale, "state_scale", torch.float32, (H, P))
    _need(cb_scale, "cb_scale", torch.float32, (G,))
    if D is not None:
        _need(D, "D", torch.float32, (H,))
    if corr is not None:
        _need(corr, "corr", torch.float32, (H, P))
    if init_state_q is not None:
        _need(init_state_q, "init_state_q", torch.int8, (B, H, P, N))
    if hand_off_timeouts is not None:
        _need(hand_off_timeouts, "hand_off_timeouts", torch.int32, (1,))
    dev = x.device
    y_dtype = x.dtype if y_dtype is None else y_dtype
    if y is None:
        y = torch.empty((B, L, H, P), dtype=y_dtype, device=dev)
    _need(y, "y", y_dtype, (B, L, H, P))
    d = dims(B, L, H, G, P, N, chunk)
    if not _noalloc:
        need = workspace_size(d)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        _need(workspace, "workspace", torch.uint8)
    elif workspace is not None:
        raise ValueError("ssd_chunk_scan_noalloc takes no workspace")
    a = ScanArgs()
    a.x, a.x_dtype = _ptr(x), _fdt(x)
    a.dt, a.dt_softplus, a.A = _ptr(dt), int(dt_softplus), _ptr(A)
    if Bq is not None:
        a.Bq, a.Cq = _ptr(Bq), _ptr(Cq)
    else:
        a.B, a.C, a.bc_dtype = _ptr(Bsrc), _ptr(Csrc), _fdt(Bsrc)
    a.B_scale, a.C_scale = _ptr(B_scale), _ptr(C_scale)
    a.c_per_token = int(c_per_token)
    a.D, a.corr = _ptr(D), _ptr(corr)
    a.xs_scale, a.xs_per_head = _ptr(xs_scale), int(xs_per_head)
    a.state_scale, a.cb_scale = _ptr(state_scale), _ptr(cb_scale)
    a.decay_shift, a.shift_round = int(decay_shift), int(shift_round)
    a.init_state_q = _ptr(init_state_q)
    a.y, a.y_dtype = _ptr(y), _fdt(y)
    out: Dict[str, torch.Tensor] = {"y": y}
    if final_state:
        out["final_state_q"] = torch.empty((B, H, P, N), dtype=torch.int8, device=dev)
        out["final_state"] = torch.empty((B, H, P, N), dtype=torch.float32, device=dev)
        a.final_state_q = _ptr(out["final_state_q"])
        a.final_state = _ptr(out["final_state"])
    c = L // chunk if chunk else 0
    for name in taps:
        dty, shp = TAPS[name]
        t = torch.zeros(shp(B, L, H, P, G, N, chunk, c), dtype=dty, device=dev)
        out[name] = t
        setattr(a, name, _ptr(t))
    if workspace is not None:
        a.workspace, a.workspace_bytes = _ptr(workspace), workspace.numel()
    if stage_events is not None:
        a.stage_events = ctypes.cast(stage_events, ctypes.c_void_p)
    a.path = PATHS[path]
    a.hand_off_timeouts = _ptr(hand_off_timeouts)
    if hand_off_timeouts is not None:
        out["hand_off_timeouts"] = hand_off_timeouts
    if _noalloc:
        st = lib().ssdi8_ssd_chunk_scan_noalloc(ctypes.byref(d), ctypes.byref(a), _stream(stream))
        _check(st, "ssdi8_ssd_chunk_scan_noalloc")
    else:
        st = lib().ssdi8_ssd_chunk_scan(ctypes.byref(d), ctypes.byref(a), _stream(stream))
        _check(st, "ssdi8_ssd_chunk_scan")
    return out


def ssd_chunk_scan_noalloc(*args, **kw) -> Dict[str, torch.Tensor]:
    """ssdi8_ssd_chunk_scan_noalloc: ssd_chunk_scan with the library's static per-GPU scratch
    instead of a workspace (no device allocation by the library; outputs and taps are still
    allocated here unless passed in, e.g. y=).  Workspaces above 128 MiB are refused."""
    if kw.get("workspace") is not None:
        raise ValueError("ssd_chunk_scan_noalloc takes no workspace")
    kw.pop("workspace", None)
    return ssd_chunk_scan(*args, _noalloc=True, **kw)


def ssd_chunk_scan_fp16(x: torch.Tensor, dt: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
                        C: torch.Tensor, *, D: Optional[torch.Tensor] = None,
                        dt_softplus: bool = True, chunk: int = CHUNK,
                        init_state: Optional[torch.Tensor] = None,
                        y_dtype: Optional[torch.dtype] = None, final_state: bool = True,
                        workspace: Optional[torch.Tensor] = None,
                        y: Optional[torch.Tensor] = None, stage_events=None,
                        stream=None) -> Dict[str, torch.Tensor]:
    """The unquantized FP16 SSD layer (ssdi8_ssd_chunk_scan_fp16), the baseline of the INT8
    path.  x (B,L,H,P), dt (B,L,H), A (H), B/C (B,L,G,N) fp16 or fp32, D (H), init_state
    (B,H,P,N) fp32.  Returns y and, with final_state, the fp32 final state."""
    _need(x, "x")
    Bt, L, H, P = x.shape
    _need(B, "B")
    G, N = B.shape[2], B.shape[3]
    _need(B, "B", B.dtype, (Bt, L, G, N))
    _need(C, "C", B.dtype, (Bt, L, G, N))
    _need(dt, "dt", torch.float32, (Bt, L, H))
    _need(A, "A", torch.float32, (H,))
    if D is not None:
        _need(D, "D", torch.float32, (H,))
    if init_state is not None:
        _need(init_state, "init_state", torch.float32, (Bt, H, P, N))
    dev = x.device
    y_dtype = x.dtype if y_dtype is None else y_dtype
    if y is None:
        y = torch.empty((Bt, L, H, P), dtype=y_dtype, device=dev)
    _need(y, "y", y_dtype, (Bt, L, H, P))
    d = dims(Bt, L, H, G, P, N, chunk)
    need = lib().ssdi8_fp16_workspace_size(ctypes.byref(d))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    a = Fp16Args()
    a.x, a.x_dtype = _ptr(x), _fdt(x)
    a.dt, a.dt_softplus, a.A = _ptr(dt), int(dt_softplus), _ptr(A)
    a.B, a.C, a.bc_dtype = _ptr(B), _ptr(C), _fdt(B)
    a.D, a.init_state = _ptr(D), _ptr(init_state)
    a.y, a.y_dtype = _ptr(y), _fdt(y)
    out: Dict[str, torch.Tensor] = {"y": y}
    if final_state:
        out["final_state"] = torch.empty((Bt, H, P, N), dtype=torch.float32, device=dev)
        a.final_state = _ptr(out["final_state"])
    if workspace is not None:
        a.workspace, a.workspace_bytes = _ptr(workspace), workspace.numel()
    if stage_events is not None:
        a.stage_events = ctypes.cast(stage_events, ctypes.c_void_p)
    st = lib().ssdi8_ssd_chunk_scan_fp16(ctypes.byref(d), ctypes.byref(a), _stream(stream))
    _check(st, "ssdi8_ssd_chunk_scan_fp16")
    return out


def uses_single_pass(d: Dims, x_dtype: torch.dtype, path: str = "auto", taps=()) -> bool:
    """Whether ssd_chunk_scan on these sizes runs the single-pass kernel (ssdi8_uses_single_pass)."""
    a = ScanArgs()
    a.x_dtype = F16 if x_dtype == torch.float16 else F32
    a.path = PATHS[path]
    for name in taps:
        setattr(a, name, 16)      # a non-NULL tap pointer (only its presence matters here)
    return bool(lib().ssdi8_uses_single_pass(ctypes.byref(d), ctypes.byref(a)))


def mfma_peak(kind: str = "int8", iters: int = 20000, blocks: int = 1024, reps: int = 3) -> float:
    """Measured MFMA rate of this GPU (ops/s; ssdi8_mfma_probe), best of `reps` launches."""
    out = torch.empty(blocks * 256, dtype=torch.int32 if kind == "int8" else torch.float32,
                      device="cuda")
    ops = ctypes.c_int64()
    k = 0 if kind == "int8" else 1
    best = 0.0
    for _ in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        st = lib().ssdi8_mfma_probe(k, iters, blocks, _ptr(out), ctypes.byref(ops), _stream(None))
        e1.record()
        _check(st, "ssdi8_mfma_probe")
        torch.cuda.synchronize()
        best = max(best, ops.value / (e0.elapsed_time(e1) * 1e-3))
    return best


def fp16_workspace_size(d: Dims) -> int:
    return int(lib().ssdi8_fp16_workspace_size(ctypes.byref(d)))


def calibrate(x: torch.Tensor, dt: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
              C: torch.Tensor, *, D: Optional[torch.Tensor] = None, dt_softplus: bool = True,
              chunk: int = CHUNK, xs_per_head: bool = False, eta: float = 0.15,
              decay_shift: int = 7, shift_round: bool = True,
              workspace: Optional[torch.Tensor] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Static steps and the per-channel mean correction from one calibration draw
    (ssdi8_calibrate).  Returns alpha_B, alpha_C (G), alpha_Xs (H,P) or (H), alpha_S (H,P),
    alpha_CB (G) and corr (H,P), fp32 on the device of x."""
    _need(x, "x")
    Bt, L, H, P = x.shape
    _need(B, "B")
    G, N = B.shape[2], B.shape[3]
    _need(B, "B", B.dtype, (Bt, L, G, N))
    _need(C, "C", B.dtype, (Bt, L, G, N))
    _need(dt, "dt", torch.float32, (Bt, L, H))
    _need(A, "A", torch.float32, (H,))
    if D is not None:
        _need(D, "D", torch.float32, (H,))
    dev = x.device
    d = dims(Bt, L, H, G, P, N, chunk)
    need = lib().ssdi8_calibrate_workspace_size(ctypes.byref(d))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(s, dtype=torch.float32, device=dev)
    out = {"alpha_B": f32(G), "alpha_C": f32(G),
           "alpha_Xs": f32(H) if xs_per_head else f32(H, P), "alpha_S": f32(H, P),
           "alpha_CB": f32(G), "corr": f32(H, P)}
    a = CalibArgs()
    a.x, a.x_dtype = _ptr(x), _fdt(x)
    a.dt, a.dt_softplus, a.A = _ptr(dt), int(dt_softplus), _ptr(A)
    a.B, a.C, a.bc_dtype, a.D = _ptr(B), _ptr(C), _fdt(B), _ptr(D)
    a.xs_per_head, a.eta = int(xs_per_head), float(eta)
    a.decay_shift, a.shift_round = int(decay_shift), int(shift_round)
    a.B_scale, a.C_scale = _ptr(out["alpha_B"]), _ptr(out["alpha_C"])
    a.xs_scale, a.state_scale = _ptr(out["alpha_Xs"]), _ptr(out["alpha_S"])
    a.cb_scale, a.corr = _ptr(out["alpha_CB"]), _ptr(out["corr"])
    if workspace is not None:
        a.workspace, a.workspace_bytes = _ptr(workspace), workspace.numel()
    st = lib().ssdi8_calibrate(ctypes.byref(d), ctypes.byref(a), _stream(stream))
    _check(st, "ssdi8_calibrate")
    return out


def calibrate_workspace_size(d: Dims) -> int:
    return int(lib().ssdi8_calibrate_workspace_size(ctypes.byref(d)))


def decode_step(x: torch.Tensor, dt: torch.Tensor, A: torch.Tensor, Bq: torch.Tensor,
                Cq: torch.Tensor, B_scale: torch.Tensor, C_scale: torch.Tensor,
                xs_scale: torch.Tensor, state_scale: torch.Tensor, cb_scale: torch.Tensor,
                state_q: torch.Tensor, *, D: Optional[torch.Tensor] = None,
                corr: Optional[torch.Tensor] = None, dt_softplus: bool = True,
                decay_shift: int = 7, shift_round: bool = True,
                y_dtype: Optional[torch.dtype] = None, y: Optional[torch.Tensor] = None,
                state_f32: bool = False, stream=None) -> Dict[str, torch.Tensor]:
    """One decode token (ssdi8_decode_step): x (B,H,P), dt (B,H), Bq/Cq (B,G,N) int8, C_scale
    (G) or (B,G); state_q (B,H,P,N) int8 is updated in place.  Returns y (B,H,P) and, with
    state_f32, the dequantized new state."""
    _need(x, "x")
    B, H, P = x.shape
    _need(Bq, "Bq", torch.int8)
    G, N = Bq.shape[1], Bq.shape[2]
    _need(Bq, "Bq", torch.int8, (B, G, N))
    _need(Cq, "Cq", torch.int8, (B, G, N))
    _need(dt, "dt", torch.float32, (B, H))
    _need(A, "A", torch.float32, (H,))
    _need(B_scale, "B_scale", torch.float32, (G,))
    c_per_token = C_scale.dim() == 2
    _need(C_scale, "C_scale", torch.float32, (B, G) if c_per_token else (G,))
    xs_per_head = xs_scale.dim() == 1
    _need(xs_scale, "xs_scale", torch.float32, (H,) if xs_per_head else (H, P))
    _need(state_scale, "state_scale", torch.float32, (H, P))
    _need(cb_scale, "cb_scale", torch.float32, (G,))
    _need(state_q, "state_q", torch.int8, (B, H, P, N))
    if D is not None:
        _need(D, "D", torch.float32, (H,))
    if corr is not None:
        _need(corr, "corr", torch.float32, (H, P))
    y_dtype = x.dtype if y_dtype is None else y_dtype
    if y is None:
        y = torch.empty((B, H, P), dtype=y_dtype, device=x.device)
    _need(y, "y", y_dtype, (B, H, P))
    a = DecodeArgs()
    a.x, a.x_dtype = _ptr(x), _fdt(x)
    a.dt, a.dt_softplus, a.A = _ptr(dt), int(dt_softplus), _ptr(A)
    a.Bq, a.Cq, a.B_scale, a.C_scale = _ptr(Bq), _ptr(Cq), _ptr(B_scale), _ptr(C_scale)
    a.c_per_token = int(c_per_token)
    a.D, a.corr = _ptr(D), _ptr(corr)
    a.xs_scale, a.xs_per_head = _ptr(xs_scale), int(xs_per_head)
    a.state_scale, a.cb_scale = _ptr(state_scale), _ptr(cb_scale)
    a.decay_shift, a.shift_round = int(decay_shift), int(shift_round)
    a.state_q = _ptr(state_q)
    a.y, a.y_dtype = _ptr(y), _fdt(y)
    out: Dict[str, torch.Tensor] = {"y": y}
    if state_f32:
        out["state"] = torch.empty((B, H, P, N), dtype=torch.float32, device=x.device)
        a.state = _ptr(out["state"])
    st = lib().ssdi8_decode_step(B, H, P, G, N, ctypes.byref(a), _stream(stream))
    _check(st, "ssdi8_decode_step")
    return out


class SSDi8Layer:
    """A quantized SSD layer with static (calibrated) steps: quantize B and C once per group,
    then run the chunk scan.  Holds device copies of the parameters and a reusable workspace."""

    def __init__(self, A, D, corr, scales: Dict[str, object], *, device="cuda",
                 dt_softplus: bool = True, decay_shift: int = 7, shift_round: bool = True):
        f = lambda v: torch.as_tensor(v, dtype=torch.float32).to(device).contiguous()
        self.A, self.D = f(A), f(D)
        self.corr = None if corr is None else f(corr)
        self.alpha_B, self.alpha_C = f(scales["alpha_B"]), f(scales["alpha_C"])
        self.alpha_Xs, self.alpha_S = f(scales["alpha_Xs"]), f(scales["alpha_S"])
        self.alpha_CB = f(scales["alpha_CB"])
        self.dt_softplus, self.decay_shift, self.shift_round = dt_softplus, decay_shift, shift_round
        self.workspace: Optional[torch.Tensor] = None
        self.Bq = self.Cq = None
        self.timeouts = torch.zeros(1, dtype=torch.int32, device=device)

    def __call__(self, x, dt, B, C, *, y=None, taps=(), final_state=True, stage_events=None,
                 path="auto", quantize_in_bmm=False, stream=None, check=True):
        """quantize_in_bmm: hand B, C to ChunkBMM unquantized (one launch fewer per tensor, no
        row-major int8 copies) instead of quantizing them first with ssdi8_quantize_act.
        check: after the call, wait for the stream and raise if a single-pass hand-off wait ran
        out (skipped while the stream is being captured into a graph; `hand_off_timeouts()`
        reads the count of the latest call then)."""
        out = self._run(x, dt, B, C, y=y, taps=taps, final_state=final_state,
                        stage_events=stage_events, path=path, quantize_in_bmm=quantize_in_bmm,
                        stream=stream)
        capturing = torch.cuda.is_current_stream_capturing()
        if check and not capturing:
            n = self.hand_off_timeouts()
            if n:
                raise RuntimeError(f"ssdi8_ssd_chunk_scan: {n} single-pass hand-off wait(s) ran "
                                   "out; y and the final states of this call are unspecified")
        return out

    def hand_off_timeouts(self) -> int:
        """Waits that ran out in the latest call (synchronises with the device)."""
        return int(self.timeouts.item())

    def _run(self, x, dt, B, C, *, y, taps, final_state, stage_events, path, quantize_in_bmm,
             stream):
        Bt, L, H, P = x.shape
        G = B.shape[2]
        need = workspace_size(dims(Bt, L, H, G))
        if self.workspace is None or self.workspace.numel() < need:
            self.workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
        if quantize_in_bmm:
            return ssd_chunk_scan(x, dt, self.A, None, None, self.alpha_B, self.alpha_C,
                                  self.alpha_Xs, self.alpha_S, self.alpha_CB, D=self.D,
                                  corr=self.corr, dt_softplus=self.dt_softplus,
                                  decay_shift=self.decay_shift, shift_round=self.shift_round,
                                  taps=taps, workspace=self.workspace, y=y,
                                  final_state=final_state, stage_events=stage_events,
                                  path=path, B=B, C=C, stream=stream,
                                  hand_off_timeouts=self.timeouts)
        if self.Bq is None or self.Bq.shape != B.shape:
            self.Bq = torch.empty(B.shape, dtype=torch.int8, device=x.device)
            self.Cq = torch.empty(C.shape, dtype=torch.int8, device=x.device)
        quantize_act(B, "group", self.alpha_B, out=self.Bq, stream=stream)
        quantize_act(C, "group", self.alpha_C, out=self.Cq, stream=stream)
        return ssd_chunk_scan(x, dt, self.A, self.Bq, self.Cq, self.alpha_B, self.alpha_C,
                              self.alpha_Xs, self.alpha_S, self.alpha_CB, D=self.D,
                              corr=self.corr, dt_softplus=self.dt_softplus,
                              decay_shift=self.decay_shift, shift_round=self.shift_round,
                              taps=taps, workspace=self.workspace, y=y,
                              final_state=final_state, stage_events=stage_events,
                              path=path, stream=stream, hand_off_timeouts=self.timeouts)


# ------------------------------------------------------------------------------ timing events
class HipEvents:
    """A pool of hipEvent_t handles from the HIP runtime that PyTorch already loaded (timing
    plumbing for the per-module breakdown; the library records them on the launch stream)."""

    def __init__(self, n: int):
        torch.cuda.init()
        self._hip = ctypes.CDLL("libamdhip64.so.7")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                  ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.handles = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            if self._hip.hipEventCreate(ctypes.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.handles[i] = h
        self.n = n

    def group(self, i: int, k: int = 5):
        """Pointer to k consecutive handles starting at i (for ScanArgs.stage_events)."""
        return ctypes.cast(ctypes.byref(self.handles, i * ctypes.sizeof(ctypes.c_void_p)),
                           ctypes.POINTER(ctypes.c_void_p))

    def record(self, i: int, stream=None) -> None:
        if self._hip.hipEventRecord(self.handles[i], _stream(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, i: int, j: int) -> float:
        ms = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), self.handles[i], self.handles[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def close(self) -> None:
        for i in range(self.n):
            if self.handles[i]:
                self._hip.hipEventDestroy(self.handles[i])
                self.handles[i] = None
