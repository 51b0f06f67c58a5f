"""ctypes binding of libmap (include/map.h): argument marshalling only.

Every function takes and returns torch tensors that live on a ROCm device;
all arithmetic happens in the library's HIP kernels, enqueued on the current
torch stream.  There is no CPU fallback: if libmap.so is missing or a call
fails, an exception is raised.

Every tensor argument (inputs, reused outputs, workspaces) is checked against
the sizes the call implies -- shape, dtype, contiguity, device -- before the
library is called, and a mismatch raises ValueError or TypeError with nothing
enqueued: the kernels trust the shapes they are given.
"""
import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmap.so")

(MAP_OK, MAP_ERR_INVALID_ARG, MAP_ERR_UNSUPPORTED, MAP_ERR_WORKSPACE, MAP_ERR_HIP, MAP_ERR_TOO_LARGE,
 MAP_ERR_NONFINITE) = range(7)
MAP_PRUNE_NOALLOC_MAX_BYTES = 96 << 20
MAP_F32, MAP_BF16 = 0, 1
MAP_MAX_BATCH, MAP_MAX_N, MAP_MAX_K = 64, 16384, 1024

# Every symbol include/map.h declares.
EXPORTS = (
    "map_status_string", "map_version", "map_score_workspace", "map_similarity_workspace",
    "map_select_workspace", "map_prune_workspace", "map_workspace_bytes", "map_score", "map_similarity", "map_select",
    "map_prune", "map_prune_assemble", "map_prune_noalloc", "map_assemble", "map_teacher_workspace", "map_teacher", "map_set_subset_tokens",
    "map_train_workspace", "map_train_step", "map_decoder_workspace", "map_decoder_layer",
    "map_selection_status", "map_set_select_images_per_launch", "map_set_finite_check", "map_timing_enable",
    "map_timing_read",
    "map_timing_reset",
)


class map_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")] + \
               [("D", ctypes.c_int32), ("D_h", ctypes.c_int32), ("d_p", ctypes.c_int32),
                ("rope_theta", ctypes.c_float)]


class map_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")]


class map_decoder_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")] + \
               [("d", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ff", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("eps", ctypes.c_float)]


class map_select_params(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("K0", ctypes.c_int32), ("tau", ctypes.c_float)]


_P, _I, _SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
_SIGS = {
    "map_status_string": (ctypes.c_char_p, [_I]),
    "map_version": (_I, []),
    "map_score_workspace": (_SZ, [_I, _I, _I, _I, ctypes.POINTER(map_weights)]),
    "map_similarity_workspace": (_SZ, [_I, _I, _I, _I]),
    "map_select_workspace": (_SZ, [_I, _I, _I]),
    "map_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I, ctypes.POINTER(map_weights), _I]),
    "map_prune_workspace": (_SZ, [_I, _I, _I, _I, ctypes.POINTER(map_weights), _I]),
    "map_score": (_I, [ctypes.POINTER(map_weights), _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "map_similarity": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _SZ, _P]),
    "map_select": (_I, [_I, _I, _P, _P, _P, map_select_params, _P, _P, _P, _P, _SZ, _P]),
    "map_prune": (_I, [ctypes.POINTER(map_weights), _I, _I, _I, _P, _P, _P, _P, _P,
                       map_select_params, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "map_prune_assemble": (_I, [ctypes.POINTER(map_weights), _I, _I, _I, _P, _P, _P, _P, _P,
                                map_select_params, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "map_prune_noalloc": (_I, [ctypes.POINTER(map_weights), _I, _I, _I, _P, _P, _P, _P, _P,
                               map_select_params, _P, _P, _P, _P, _P, _P, _P]),
    "map_assemble": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P]),
    "map_teacher_workspace": (_SZ, [_I, _I, _I]),
    "map_teacher": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "map_train_workspace": (_SZ, [_I, _I, _I, _I, ctypes.POINTER(map_weights)]),
    "map_train_step": (_I, [ctypes.POINTER(map_weights), _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P,
                            ctypes.POINTER(map_grads), _P, _SZ, _P]),
    "map_decoder_workspace": (_SZ, [_I, ctypes.POINTER(map_decoder_weights)]),
    "map_decoder_layer": (_I, [ctypes.POINTER(map_decoder_weights), _I, _I, _P, _P, _P, _P, _P, _SZ, _P]),
    "map_set_subset_tokens": (_I, [_I]),
    "map_selection_status": (_I, [_P, _P, _P]),
    "map_set_select_images_per_launch": (_I, [_I]),
    "map_set_finite_check": (_I, [_I]),
    "map_timing_enable": (_I, [_I]),
    "map_timing_read": (_I, [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                             ctypes.POINTER(ctypes.c_int), _I]),
    "map_timing_reset": (None, []),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libmap (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_06411_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


class MapError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = lib().map_status_string(status).decode()
        super().__init__(f"{where}: {msg} (status {status})")
        self.status = status


def _check(status: int, where: str):
    if status != MAP_OK:
        raise MapError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MAP_BF16
    if t.dtype == torch.float32:
        return MAP_F32
    raise TypeError(f"unsupported dtype {t.dtype}; use torch.float32 or torch.bfloat16")


def _need(t: torch.Tensor, name: str, shape, dtype, device):
    """Raise unless t is a contiguous `dtype` tensor of `shape` on `device`
    (device None: only checked to be a GPU device, by _on_gpu)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, got "
                         f"{t.dtype} {tuple(t.shape)}{'' if t.is_contiguous() else ' (not contiguous)'}")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: expected a tensor on {device}, got one on {t.device}")


def _on_gpu(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a ROCm device, got {t.device}")
    return t.device


def _dims(t: torch.Tensor, name: str, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dim() != ndim:
        raise ValueError(f"{name}: expected {ndim} dimensions, got shape {tuple(t.shape)}")
    return tuple(t.shape)


def _need_ws(ws: Optional[torch.Tensor], nbytes: int, device, name="workspace"):
    if nbytes == 0:
        return
    if ws is None or not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous uint8 buffer")
    if ws.numel() < nbytes or ws.device != device or ws.data_ptr() % 256:
        raise ValueError(f"{name}: needs {nbytes} bytes, 256-byte aligned, on {device}")


def _workspace(nbytes: int, device) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + nbytes]


@dataclass
class PredictorWeights:
    """Predictor parameters on the device (torch.nn.Linear layout)."""
    w1_v: torch.Tensor
    b1_v: torch.Tensor
    w2_v: torch.Tensor
    b2_v: torch.Tensor
    w_k: torch.Tensor
    w1_t: torch.Tensor
    b1_t: torch.Tensor
    w2_t: torch.Tensor
    b2_t: torch.Tensor
    w_q: torch.Tensor
    rope_theta: float = 10000.0

    @property
    def D(self):
        return self.w1_v.shape[1]

    @property
    def D_h(self):
        return self.w1_v.shape[0]

    @property
    def d_p(self):
        return self.w_k.shape[0]

    @property
    def dtype(self):
        return self.w1_v.dtype

    def check(self, D: int, dtype, device):
        """Raise unless every weight has the shape the predictor implies for
        feature width D (torch.nn.Linear layout), the call's dtype and device."""
        _dims(self.w1_v, "w1_v", 2)
        _dims(self.w_k, "w_k", 2)
        Dh, dp = self.D_h, self.d_p
        shapes = {"w1_v": (Dh, D), "b1_v": (Dh,), "w2_v": (Dh, Dh), "b2_v": (Dh,), "w_k": (dp, Dh),
                  "w1_t": (Dh, D), "b1_t": (Dh,), "w2_t": (Dh, Dh), "b2_t": (Dh,), "w_q": (dp, Dh)}
        for n, shape in shapes.items():
            _need(getattr(self, n), f"weight {n}", shape, dtype, device)

    def struct(self) -> map_weights:
        s = map_weights()
        for n in ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q"):
            t = getattr(self, n)
            if not t.is_contiguous() or t.dtype != self.dtype:
                raise ValueError(f"weight {n} must be contiguous {self.dtype}")
            setattr(s, n, t.data_ptr())
        s.D, s.D_h, s.d_p, s.rope_theta = self.D, self.D_h, self.d_p, float(self.rope_theta)
        return s


def _offsets(t_off, B: Optional[int] = None) -> (ctypes.Array, int):
    vals = [int(x) for x in (t_off.tolist() if hasattr(t_off, "tolist") else t_off)]
    if B is not None and len(vals) != B + 1:
        raise ValueError(f"offsets need B + 1 = {B + 1} entries, got {len(vals)}")
    if len(vals) < 2 or vals[0] != 0 or any(b <= a for a, b in zip(vals, vals[1:])):
        raise ValueError("offsets must start at 0 and increase strictly")
    arr = (ctypes.c_int32 * len(vals))(*vals)
    return arr, vals[-1]


def _check_features(w: PredictorWeights, V, pos_v, T, pos_t, t_off):
    """The inputs of map_score / map_prune: returns (B, N, D, sumM, offsets, device)."""
    B, N, D = _dims(V, "V", 3)
    _dtype_code(V)
    offs, sumM = _offsets(t_off, B)
    _need(V, "V", (B, N, D), V.dtype, None)
    dev = V.device  # (checked to be a GPU device before the library is called)
    _need(pos_v, "pos_v", (B, N), torch.int32, dev)
    _need(T, "T", (sumM, D), V.dtype, dev)
    _need(pos_t, "pos_t", (sumM,), torch.int32, dev)
    w.check(D, V.dtype, dev)
    return B, N, D, sumM, offs, dev


def map_score(w: PredictorWeights, V: torch.Tensor, pos_v: torch.Tensor, T: torch.Tensor,
              pos_t: torch.Tensor, t_off: Sequence[int], p_out: Optional[torch.Tensor] = None):
    """Predicted attention p_hat [B, N] (Eq. (3))."""
    B, N, D, sumM, offs, dev = _check_features(w, V, pos_v, T, pos_t, t_off)
    if p_out is None:
        p_out = torch.empty(B, N, dtype=torch.float32, device=dev)
    _need(p_out, "p_out", (B, N), torch.float32, dev)
    _on_gpu(V, "V")
    ws_struct = w.struct()
    dt = _dtype_code(V)
    nbytes = lib().map_score_workspace(dt, B, N, sumM, ctypes.byref(ws_struct))
    if nbytes == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_score_workspace")
    ws = _workspace(nbytes, dev)
    _check(lib().map_score(ctypes.byref(ws_struct), dt, B, N, _ptr(V), _ptr(pos_v), _ptr(T),
                           _ptr(pos_t), offs, _ptr(p_out), _ptr(ws), nbytes, _stream(dev)),
           "map_score")
    return p_out


def map_similarity(V: torch.Tensor, S_out: Optional[torch.Tensor] = None,
                   norms_out: Optional[torch.Tensor] = None, norms_only: bool = False):
    """Cosine similarity S [B, N, N] and row norms [B, N] of the visual tokens.
    With norms_only the library forms the norms alone and S is None."""
    B, N, D = _dims(V, "V", 3)
    dt = _dtype_code(V)
    _need(V, "V", (B, N, D), V.dtype, None)
    dev = V.device
    if S_out is None and not norms_only:
        S_out = torch.empty(B, N, N, dtype=torch.float32, device=dev)
    if norms_out is None:
        norms_out = torch.empty(B, N, dtype=torch.float32, device=dev)
    if norms_only:
        S_out = None
    else:
        _need(S_out, "S_out", (B, N, N), torch.float32, dev)
    _need(norms_out, "norms_out", (B, N), torch.float32, dev)
    _on_gpu(V, "V")
    nbytes = lib().map_similarity_workspace(dt, B, N, D)
    ws = _workspace(nbytes, dev)
    _check(lib().map_similarity(dt, B, N, D, _ptr(V), _ptr(S_out), _ptr(norms_out), _ptr(ws),
                                nbytes, _stream(dev)), "map_similarity")
    return S_out, norms_out


def map_select(p: torch.Tensor, S: torch.Tensor, norms: torch.Tensor, K: int, K0: int,
               tau: float = 1e-2, idx_out=None, order_out=None, gain_out=None):
    """Diversity-aware selection (Eq. (4)): returns (idx ascending, order, gain), each [B, K]."""
    B, N = _dims(p, "p", 2)
    _need(p, "p", (B, N), torch.float32, None)
    dev = p.device
    _need(S, "S", (B, N, N), torch.float32, dev)
    _need(norms, "norms", (B, N), torch.float32, dev)
    idx_out = torch.empty(B, K, dtype=torch.int32, device=dev) if idx_out is None else idx_out
    order_out = torch.empty(B, K, dtype=torch.int32, device=dev) if order_out is None else order_out
    gain_out = torch.empty(B, K, dtype=torch.float32, device=dev) if gain_out is None else gain_out
    _need(idx_out, "idx_out", (B, K), torch.int32, dev)
    _need(order_out, "order_out", (B, K), torch.int32, dev)
    _need(gain_out, "gain_out", (B, K), torch.float32, dev)
    _on_gpu(p, "p")
    nbytes = lib().map_select_workspace(B, N, K)
    if nbytes == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_select_workspace")
    ws = _workspace(nbytes, dev)
    sp = map_select_params(K, K0, tau)
    _check(lib().map_select(B, N, _ptr(p), _ptr(S), _ptr(norms), sp, _ptr(idx_out), _ptr(order_out),
                            _ptr(gain_out), _ptr(ws), nbytes, _stream(dev)), "map_select")
    return idx_out, order_out, gain_out


class PruneWorkspace:
    """Reusable workspace for repeated map_prune calls of one shape."""

    def __init__(self, w: PredictorWeights, V: torch.Tensor, t_off, K: int):
        B, N, D = _dims(V, "V", 3)
        offs, sumM = _offsets(t_off, B)
        dev = _on_gpu(V, "V")
        self.nbytes = lib().map_prune_workspace(_dtype_code(V), B, N, sumM, ctypes.byref(w.struct()), K)
        if self.nbytes == 0:
            raise MapError(MAP_ERR_INVALID_ARG, "map_prune_workspace")
        self.buf = _workspace(self.nbytes, dev)
        self.device = dev

    def status(self) -> int:
        """The selection status word of the last call on this workspace
        (0: completed; 1: a barrier wait expired).  Synchronises the stream."""
        return selection_status(self.buf)


def map_prune(w: PredictorWeights, V: torch.Tensor, pos_v: torch.Tensor, T: torch.Tensor,
              pos_t: torch.Tensor, t_off: Sequence[int], K: int, K0: int, tau: float = 1e-2,
              out: Optional[dict] = None, workspace: Optional[PruneWorkspace] = None):
    """Fused score + similarity + selection + gather.  Returns a dict with
    idx, V_out, pos_out, p, order and gain (the given `out` tensors are
    filled in place)."""
    B, N, D, sumM, offs, dev = _check_features(w, V, pos_v, T, pos_t, t_off)
    o = dict(out or {})
    o.setdefault("idx", torch.empty(B, K, dtype=torch.int32, device=dev))
    o.setdefault("V_out", torch.empty(B, K, D, dtype=V.dtype, device=dev))
    o.setdefault("pos_out", torch.empty(B, K, dtype=torch.int32, device=dev))
    o.setdefault("p", torch.empty(B, N, dtype=torch.float32, device=dev))
    o.setdefault("order", torch.empty(B, K, dtype=torch.int32, device=dev))
    o.setdefault("gain", torch.empty(B, K, dtype=torch.float32, device=dev))
    for name, shape, dtype in (("idx", (B, K), torch.int32), ("V_out", (B, K, D), V.dtype),
                               ("pos_out", (B, K), torch.int32), ("p", (B, N), torch.float32),
                               ("order", (B, K), torch.int32), ("gain", (B, K), torch.float32)):
        _need(o[name], f"out[{name!r}]", shape, dtype, dev)
    _on_gpu(V, "V")
    if workspace is None:
        workspace = PruneWorkspace(w, V, t_off, K)
    need = lib().map_prune_workspace(_dtype_code(V), B, N, sumM, ctypes.byref(w.struct()), K)
    if need == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_prune_workspace")
    _need_ws(workspace.buf, need, dev)
    ws_struct = w.struct()
    sp = map_select_params(K, K0, tau)
    _check(lib().map_prune(ctypes.byref(ws_struct), _dtype_code(V), B, N, _ptr(V), _ptr(pos_v),
                           _ptr(T), _ptr(pos_t), offs, sp, _ptr(o["idx"]), _ptr(o["V_out"]),
                           _ptr(o["pos_out"]), _ptr(o["p"]), _ptr(o["order"]), _ptr(o["gain"]),
                           _ptr(workspace.buf), workspace.nbytes, _stream(dev)), "map_prune")
    return o


def map_prune_assemble(w: PredictorWeights, V: torch.Tensor, pos_v: torch.Tensor, T: torch.Tensor,
                       pos_t: torch.Tensor, t_off: Sequence[int], K: int, K0: int, tau: float = 1e-2,
                       out: Optional[dict] = None, workspace: Optional[PruneWorkspace] = None):
    """map_prune that writes the language model's layer-0 input directly:
    returns a dict with X [B K + sum M, D] (each image's kept rows in original
    order, then its question rows), pos_x, idx, p, order and gain."""
    B, N, D, sumM, offs, dev = _check_features(w, V, pos_v, T, pos_t, t_off)
    o = dict(out or {})
    o.setdefault("idx", torch.empty(B, K, dtype=torch.int32, device=dev))
    o.setdefault("X", torch.empty(B * K + sumM, D, dtype=V.dtype, device=dev))
    o.setdefault("pos_x", torch.empty(B * K + sumM, dtype=torch.int32, device=dev))
    o.setdefault("p", torch.empty(B, N, dtype=torch.float32, device=dev))
    o.setdefault("order", torch.empty(B, K, dtype=torch.int32, device=dev))
    o.setdefault("gain", torch.empty(B, K, dtype=torch.float32, device=dev))
    for name, shape, dtype in (("idx", (B, K), torch.int32), ("X", (B * K + sumM, D), V.dtype),
                               ("pos_x", (B * K + sumM,), torch.int32), ("p", (B, N), torch.float32),
                               ("order", (B, K), torch.int32), ("gain", (B, K), torch.float32)):
        _need(o[name], f"out[{name!r}]", shape, dtype, dev)
    _on_gpu(V, "V")
    if workspace is None:
        workspace = PruneWorkspace(w, V, t_off, K)
    need = lib().map_prune_workspace(_dtype_code(V), B, N, sumM, ctypes.byref(w.struct()), K)
    if need == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_prune_workspace")
    _need_ws(workspace.buf, need, dev)
    ws_struct = w.struct()
    _check(lib().map_prune_assemble(ctypes.byref(ws_struct), _dtype_code(V), B, N, _ptr(V), _ptr(pos_v), _ptr(T),
                                    _ptr(pos_t), offs, map_select_params(K, K0, tau), _ptr(o["idx"]), _ptr(o["X"]),
                                    _ptr(o["pos_x"]), _ptr(o["p"]), _ptr(o["order"]), _ptr(o["gain"]),
                                    _ptr(workspace.buf), workspace.nbytes, _stream(dev)), "map_prune_assemble")
    return o


def map_assemble(V_out: torch.Tensor, pos_out: torch.Tensor, T: torch.Tensor, pos_t: torch.Tensor,
                 t_off: Sequence[int]):
    """The layer-0 input after pruning: per image its K kept rows, then its
    question rows, packed; returns (X [B K + sum M][D], positions)."""
    B, K, D = _dims(V_out, "V_out", 3)
    _dtype_code(V_out)
    offs, sumM = _offsets(t_off, B)
    _need(V_out, "V_out", (B, K, D), V_out.dtype, None)
    dev = V_out.device
    _need(pos_out, "pos_out", (B, K), torch.int32, dev)
    _need(T, "T", (sumM, D), V_out.dtype, dev)
    _need(pos_t, "pos_t", (sumM,), torch.int32, dev)
    _on_gpu(V_out, "V_out")
    X = torch.empty(B * K + sumM, D, dtype=V_out.dtype, device=dev)
    pos = torch.empty(B * K + sumM, dtype=torch.int32, device=dev)
    _check(lib().map_assemble(_dtype_code(V_out), B, K, D, _ptr(V_out), _ptr(pos_out), _ptr(T), _ptr(pos_t), offs,
                              _ptr(X), _ptr(pos), _stream(dev)), "map_assemble")
    return X, pos


def map_teacher(A: torch.Tensor, A_ref: torch.Tensor, m_off: Sequence[int], L: int, H: int, N: int, M_ref: int,
                n_top: int = 1, out: Optional[dict] = None) -> dict:
    """Teacher selection (Eq. (1)-(2), QCTS-n).  A holds sample b's
    [L][H][M_b][N] attention back to back (M_b from m_off), A_ref is
    [B][L][H][M_ref][N]; both contiguous, same dtype.  Returns p, p_ref
    [B, L, N], js [B, L] (float64), layers [B, n_top] and teacher [B, N];
    ``out`` (a previous result) is written in place when given."""
    offs, sumM = _offsets(m_off)
    B = len(offs) - 1
    dt = _dtype_code(A)
    if A.numel() != L * H * sumM * N or A_ref.numel() != B * L * H * M_ref * N:
        raise ValueError("A or A_ref does not hold the sizes given")
    if A_ref.dtype != A.dtype or not A.is_contiguous() or not A_ref.is_contiguous():
        raise ValueError("A and A_ref must be contiguous and of one dtype")
    dev = A.device
    if A_ref.device != dev:
        raise ValueError("A and A_ref must be on one device")
    if not 1 <= n_top <= L:
        raise ValueError(f"n_top must lie in [1, L = {L}]")
    _on_gpu(A, "A")
    if out is None:
        out = dict(p=torch.empty(B, L, N, dtype=torch.float32, device=dev),
                   p_ref=torch.empty(B, L, N, dtype=torch.float32, device=dev),
                   js=torch.empty(B, L, dtype=torch.float64, device=dev),
                   layers=torch.empty(B, n_top, dtype=torch.int32, device=dev),
                   teacher=torch.empty(B, N, dtype=torch.float32, device=dev))
        nbytes = lib().map_teacher_workspace(B, L, N)
        out["_ws"] = _workspace(nbytes, dev)
    for name, shape, dtype in (("p", (B, L, N), torch.float32), ("p_ref", (B, L, N), torch.float32),
                               ("js", (B, L), torch.float64), ("layers", (B, n_top), torch.int32),
                               ("teacher", (B, N), torch.float32)):
        _need(out[name], f"out[{name!r}]", shape, dtype, dev)
    ws = out.get("_ws")
    _need_ws(ws, lib().map_teacher_workspace(B, L, N), dev, "out['_ws']")
    _check(lib().map_teacher(dt, B, L, H, N, _ptr(A), offs, _ptr(A_ref), M_ref, n_top, _ptr(out["p"]),
                             _ptr(out["p_ref"]), _ptr(out["js"]), _ptr(out["layers"]), _ptr(out["teacher"]),
                             _ptr(ws), 0 if ws is None else ws.numel(), _stream(dev)), "map_teacher")
    return out


def set_subset_tokens(n: int):
    """map_prune's candidate subset: n < 0 never, 0 automatic, n > 0 that
    many tokens.  Process-wide; workspaces sized before a change may be too
    small after it (map_prune then reports a workspace error)."""
    _check(lib().map_set_subset_tokens(int(n)), "map_set_subset_tokens")


GRAD_NAMES = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")


class TrainWorkspace:
    """Reusable workspace for repeated map_train_step calls of one shape."""

    def __init__(self, w: PredictorWeights, V: torch.Tensor, t_off):
        B, N, D = _dims(V, "V", 3)
        offs, sumM = _offsets(t_off, B)
        dev = _on_gpu(V, "V")
        self.nbytes = lib().map_train_workspace(_dtype_code(V), B, N, sumM, ctypes.byref(w.struct()))
        if self.nbytes == 0:
            raise MapError(MAP_ERR_INVALID_ARG, "map_train_workspace")
        self.buf = _workspace(self.nbytes, dev)


def map_train_step(w: PredictorWeights, V: torch.Tensor, pos_v: torch.Tensor, T: torch.Tensor,
                   pos_t: torch.Tensor, t_off: Sequence[int], p_teacher: torch.Tensor,
                   grads: Optional[dict] = None, p_out: Optional[torch.Tensor] = None,
                   workspace: Optional[TrainWorkspace] = None):
    """One predictor training step: the KL divergence from the teacher rows
    p_teacher [B, N] to p_hat (float32 per image) and the float32 gradients of
    the batch mean with respect to every predictor parameter (a dict keyed
    like PredictorWeights' fields, written in place when given).
    Returns (loss [B], p_hat [B, N], grads)."""
    B, N, D, sumM, offs, dev = _check_features(w, V, pos_v, T, pos_t, t_off)
    _need(p_teacher, "p_teacher", (B, N), torch.float32, dev)
    if grads is None:
        grads = {n: torch.empty(tuple(getattr(w, n).shape), dtype=torch.float32, device=dev) for n in GRAD_NAMES}
    for n in GRAD_NAMES:
        _need(grads[n], f"grads[{n!r}]", tuple(getattr(w, n).shape), torch.float32, dev)
    if p_out is None:
        p_out = torch.empty(B, N, dtype=torch.float32, device=dev)
    _need(p_out, "p_out", (B, N), torch.float32, dev)
    loss = torch.empty(B, dtype=torch.float32, device=dev)
    _on_gpu(V, "V")
    if workspace is None:
        workspace = TrainWorkspace(w, V, t_off)
    need = lib().map_train_workspace(_dtype_code(V), B, N, sumM, ctypes.byref(w.struct()))
    if need == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_train_workspace")
    _need_ws(workspace.buf, need, dev)
    gs = map_grads(*[grads[n].data_ptr() for n in GRAD_NAMES])
    ws_struct = w.struct()
    _check(lib().map_train_step(ctypes.byref(ws_struct), _dtype_code(V), B, N, _ptr(V), _ptr(pos_v), _ptr(T),
                                _ptr(pos_t), offs, _ptr(p_teacher), _ptr(loss), _ptr(p_out), ctypes.byref(gs),
                                _ptr(workspace.buf), workspace.nbytes, _stream(dev)), "map_train_step")
    return loss, p_out, grads


@dataclass
class DecoderWeights:
    """One LLaMA-style decoder layer on the device (bf16, torch.nn.Linear
    layout): w_qkv stacks W_q, W_k, W_v by rows, w_gate_up the gate's rows
    then the up rows."""
    attn_norm: torch.Tensor
    w_qkv: torch.Tensor
    w_o: torch.Tensor
    ffn_norm: torch.Tensor
    w_gate_up: torch.Tensor
    w_down: torch.Tensor
    n_heads: int
    rope_theta: float = 10000.0
    eps: float = 1e-6

    def struct(self, device) -> map_decoder_weights:
        d = self.w_o.shape[0]
        ff = self.w_down.shape[1]
        shapes = {"attn_norm": (d,), "w_qkv": (3 * d, d), "w_o": (d, d), "ffn_norm": (d,),
                  "w_gate_up": (2 * ff, d), "w_down": (d, ff)}
        s = map_decoder_weights()
        for n, shape in shapes.items():
            _need(getattr(self, n), f"decoder weight {n}", shape, torch.bfloat16, device)
            setattr(s, n, getattr(self, n).data_ptr())
        s.d, s.n_heads, s.ff = d, self.n_heads, ff
        s.head_dim = d // self.n_heads
        s.rope_theta, s.eps = float(self.rope_theta), float(self.eps)
        return s


def map_decoder_layer(w: DecoderWeights, X: torch.Tensor, pos: torch.Tensor, seq_off: Sequence[int],
                      out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """One decoder layer's prefill over packed sequences X [R, d] (sequence b
    is rows seq_off[b] .. seq_off[b+1]-1, causal within it; pos [R] the rows'
    positional indices).  Returns Y [R, d]."""
    R, d = _dims(X, "X", 2)
    offs, total = _offsets(seq_off)
    B = len(offs) - 1
    if total != R:
        raise ValueError(f"seq_off ends at {total}, X has {R} rows")
    _need(X, "X", (R, d), torch.bfloat16, None)
    dev = X.device
    _need(pos, "pos", (R,), torch.int32, dev)
    if out is None:
        out = torch.empty_like(X)
    _need(out, "out", (R, d), torch.bfloat16, dev)
    ws_struct = w.struct(dev)
    _on_gpu(X, "X")
    nbytes = lib().map_decoder_workspace(R, ctypes.byref(ws_struct))
    if nbytes == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_decoder_workspace")
    ws = workspace if workspace is not None else _workspace(nbytes, dev)
    _need_ws(ws, nbytes, dev)
    _check(lib().map_decoder_layer(ctypes.byref(ws_struct), MAP_BF16, B, _ptr(X), _ptr(pos), offs, _ptr(out), _ptr(ws),
                                   ws.numel(), _stream(dev)), "map_decoder_layer")
    return out


def decoder_workspace(w: DecoderWeights, R: int, device) -> torch.Tensor:
    """A reusable workspace for map_decoder_layer over R rows."""
    nbytes = lib().map_decoder_workspace(R, ctypes.byref(w.struct(device)))
    if nbytes == 0:
        raise MapError(MAP_ERR_INVALID_ARG, "map_decoder_workspace")
    return _workspace(nbytes, device)


def selection_status(ws: torch.Tensor) -> int:
    """The status word map_select / map_prune left at the start of workspace
    `ws` (0: completed; 1: a selection barrier wait expired and the call's
    indices are -1).  Copies it on the current stream and synchronises."""
    dev = _on_gpu(ws, "ws")
    word = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().map_selection_status(_ptr(ws), _ptr(word), _stream(dev)), "map_selection_status")
    return int(word.item())


def set_select_images_per_launch(n: int):
    """At most n images per persistent selection launch (n <= 0: as many as
    fit, the default).  Process-wide; for testing the multi-launch path."""
    _check(lib().map_set_select_images_per_launch(int(n)), "map_set_select_images_per_launch")


def set_finite_check(on: bool):
    """The library's finite check (a debugging aid, off by default): while
    on, each call first scans its float inputs for infinities and NaNs, waits
    for the scan and raises MapError(MAP_ERR_NONFINITE) if it finds one.
    Process-wide."""
    _check(lib().map_set_finite_check(1 if on else 0), "map_set_finite_check")


def timing_enable(on: bool = True):
    _check(lib().map_timing_enable(1 if on else 0), "map_timing_enable")


def timing_reset():
    lib().map_timing_reset()


def timing_read(cap: int = 32) -> dict:
    """{kernel name: (total ms, launches)} for the launches recorded so far."""
    names = (ctypes.c_char_p * cap)()
    ms = (ctypes.c_double * cap)()
    cnt = (ctypes.c_int * cap)()
    n = lib().map_timing_read(names, ms, cnt, cap)
    return {names[i].decode(): (ms[i], cnt[i]) for i in range(min(n, cap))}
