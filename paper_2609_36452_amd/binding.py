"""Python binding of the C ABI declared in include/rpd.h.

Argument marshalling only: torch tensors supply device memory and the
current stream; every step of the commit step runs in the HIP library
``librpd.so``. The library is loaded on first use and its absence is an
error (there is no other implementation behind these functions).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librpd.so")

DTYPE_BF16 = 0
DTYPE_F32 = 1

FLAG_CANDIDATE = 1
FLAG_HIGH_CONF = 2
FLAG_STABLE = 4
FLAG_COMMITTED = 8
FLAG_FALLBACK = 16

DEVICE_STATUS_MASKED_OVERFLOW = 1
PARAM_LAZY = 1

STATUS_NAMES = {0: "RPD_OK", 1: "RPD_ERR_NULL_POINTER", 2: "RPD_ERR_BAD_SHAPE", 3: "RPD_ERR_BAD_PARAM",
                4: "RPD_ERR_WORKSPACE_TOO_SMALL", 5: "RPD_ERR_UNSUPPORTED", 6: "RPD_ERR_HIP"}


class RpdProblem(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("B", ctypes.c_int32), ("L", ctypes.c_int32),
                ("d", ctypes.c_int32), ("V", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("hidden", ctypes.c_void_p), ("w_u", ctypes.c_void_p), ("mask", ctypes.c_void_p),
                ("max_masked", ctypes.c_int32), ("norm_weight", ctypes.c_void_p), ("norm_eps", ctypes.c_float),
                ("norm_final", ctypes.c_int32)]


class RpdParams(ctypes.Structure):
    _fields_ = [("theta_h", ctypes.c_float), ("theta_c", ctypes.c_float), ("theta_s", ctypes.c_float),
                ("w", ctypes.c_float), ("k_max", ctypes.c_int32), ("beta", ctypes.c_float),
                ("window", ctypes.c_int32), ("flags", ctypes.c_uint32), ("block", ctypes.c_int32),
                ("logit_scale", ctypes.c_float)]


_OUT_FIELDS = ["commit", "token", "entropy", "confidence", "persistence", "drop", "stability", "flags",
               "upstream_entropy", "n_commit", "layer_argmax", "layer_conf", "layer_entropy", "status"]


class RpdOutputs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _OUT_FIELDS]


@dataclass(frozen=True)
class Params:
    """Commit-rule hyperparameters (Table 4, Appendix A.6)."""
    theta_h: float = 0.9
    theta_c: float = 0.6
    theta_s: float = 3.5
    w: float = 15.0
    k_max: int = 6
    beta: float = 4.0
    window: int = 32
    block: int = 0     # 0: full RPD; > 0: RPD-block with blocks of this many positions
    logit_scale: float = 1.0   # inverse temperature of the scoring softmax
    lazy: bool = False         # lazy layerwise projection (RPD_PARAM_LAZY)

    @staticmethod
    def llada() -> "Params":
        return Params(theta_s=3.5, w=15.0)

    @staticmethod
    def dream() -> "Params":
        return Params(theta_s=2.5, w=20.0)

    @staticmethod
    def strict(K: int, beta: float = 1.0) -> "Params":
        """All K layers agree and the final probability is the peak (Eq. 4
        with w = 1, K_max >= K, theta_s = K)."""
        return Params(theta_s=float(K), w=1.0, k_max=max(K, 6), beta=beta)

    def to_c(self) -> RpdParams:
        return RpdParams(self.theta_h, self.theta_c, self.theta_s, self.w, int(self.k_max), self.beta,
                         int(self.window), PARAM_LAZY if self.lazy else 0, int(self.block),
                         float(self.logit_scale))


class RpdError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {detail}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(the commit step has no other implementation)")
        L = ctypes.CDLL(_LIB_PATH)
        L.rpd_workspace_size.restype = ctypes.c_size_t
        L.rpd_workspace_size.argtypes = [ctypes.POINTER(RpdProblem)]
        L.rpd_score_commit.restype = ctypes.c_int
        L.rpd_score_commit.argtypes = [ctypes.POINTER(RpdProblem), ctypes.POINTER(RpdParams),
                                       ctypes.POINTER(RpdOutputs), ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p]
        L.rpd_score_commit_timed.restype = ctypes.c_int
        L.rpd_score_commit_timed.argtypes = [ctypes.POINTER(RpdProblem), ctypes.POINTER(RpdParams),
                                             ctypes.POINTER(RpdOutputs), ctypes.c_void_p, ctypes.c_size_t,
                                             ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32]
        L.rpd_gate_commit.restype = ctypes.c_int
        L.rpd_gate_commit.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.POINTER(RpdParams), ctypes.POINTER(RpdOutputs), ctypes.c_void_p]
        L.rpd_status_string.restype = ctypes.c_char_p
        L.rpd_status_string.argtypes = [ctypes.c_int]
        L.rpd_last_error.restype = ctypes.c_char_p
        L.rpd_last_error.argtypes = []
        L.rpd_projection_variant.restype = ctypes.c_int32
        L.rpd_projection_variant.argtypes = [ctypes.POINTER(RpdProblem)]
        L.rpd_abi_version.restype = ctypes.c_int32
        L.rpd_abi_version.argtypes = []
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().rpd_status_string(s).decode()


def last_error() -> str:
    return lib().rpd_last_error().decode()


def abi_version() -> int:
    return int(lib().rpd_abi_version())


def _check(status: int) -> None:
    if status != 0:
        raise RpdError(status, last_error())


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def make_problem(K, B, L, d, V, dtype_code, hidden=None, w_u=None, mask=None, max_masked=-1,
                 norm_weight=None, norm_eps: float = 0.0, norm_final: bool = False) -> RpdProblem:
    nw = norm_weight if isinstance(norm_weight, (int, type(None))) else _ptr(norm_weight)
    return RpdProblem(K, B, L, d, V, dtype_code, _ptr(hidden), _ptr(w_u), _ptr(mask), int(max_masked),
                      nw, float(norm_eps), int(bool(norm_final)))


def workspace_size(K: int, B: int, L: int, d: int, V: int, dtype: torch.dtype | int,
                   max_masked: int = -1, norm: bool = False) -> int:
    code = dtype if isinstance(dtype, int) else (DTYPE_BF16 if dtype == torch.bfloat16 else DTYPE_F32)
    p = make_problem(K, B, L, d, V, code, max_masked=max_masked, norm_weight=1 if norm else None)
    return int(lib().rpd_workspace_size(ctypes.byref(p)))


PROJ_VARIANTS = {0: "bf16_s32", 1: "bf16_s64", 2: "bf16_s128", 3: "f32", 4: "bf16_big", 5: "bf16_s192",
                 6: "bf16_s256"}


def projection_variant(K: int, B: int, L: int, d: int, V: int, dtype: torch.dtype | int,
                       max_masked: int = -1) -> str:
    """Name of the projection kernel variant rpd_score_commit launches for
    this shape (rpd_projection_variant)."""
    code = dtype if isinstance(dtype, int) else (DTYPE_BF16 if dtype == torch.bfloat16 else DTYPE_F32)
    p = make_problem(K, B, L, d, V, code, max_masked=max_masked)
    v = int(lib().rpd_projection_variant(ctypes.byref(p)))
    if v < 0:
        raise RpdError(2, f"invalid shape or dtype for a plan: K={K} B={B} L={L} d={d} V={V} dtype={code}")
    return PROJ_VARIANTS[v]


def alloc_outputs(K: int, B: int, L: int, device, layer_stats: bool = False) -> dict:
    e = dict(device=device)
    o = {
        "commit": torch.empty((B, L), dtype=torch.uint8, **e),
        "token": torch.empty((B, L), dtype=torch.int32, **e),
        "entropy": torch.empty((B, L), dtype=torch.float32, **e),
        "confidence": torch.empty((B, L), dtype=torch.float32, **e),
        "persistence": torch.empty((B, L), dtype=torch.int32, **e),
        "drop": torch.empty((B, L), dtype=torch.float32, **e),
        "stability": torch.empty((B, L), dtype=torch.float32, **e),
        "flags": torch.empty((B, L), dtype=torch.uint8, **e),
        "upstream_entropy": torch.empty((B, L), dtype=torch.float32, **e),
        "n_commit": torch.empty((B,), dtype=torch.int32, **e),
        "status": torch.empty((1,), dtype=torch.int32, **e),
    }
    if layer_stats:
        o["layer_argmax"] = torch.empty((K, B, L), dtype=torch.int32, **e)
        o["layer_conf"] = torch.empty((K, B, L), dtype=torch.float32, **e)
        o["layer_entropy"] = torch.empty((K, B, L), dtype=torch.float32, **e)
    return o


def _outputs_struct(o: dict) -> RpdOutputs:
    return RpdOutputs(*[_ptr(o.get(n)) for n in _OUT_FIELDS])


def _stream_handle(stream) -> int | None:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream or None


def _check_dev(name: str, t: torch.Tensor, shape: tuple, dtypes) -> None:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class ScoreCommit:
    """A reusable call of ``rpd_score_commit`` for one problem shape: the
    outputs and the workspace are allocated once (by torch) and every
    ``__call__`` only enqueues the library's kernels."""

    def __init__(self, hidden: torch.Tensor, w_u: torch.Tensor, mask: torch.Tensor, params: Params,
                 max_masked: int | None = None, layer_stats: bool = False, norm_weight: torch.Tensor | None = None,
                 norm_eps: float = 1e-5, norm_final: bool = False):
        K, B, L, d = hidden.shape
        V = w_u.shape[0]
        code = _dtype_code(hidden)
        _check_dev("hidden", hidden, (K, B, L, d), (hidden.dtype,))
        _check_dev("w_u", w_u, (V, d), (hidden.dtype,))
        _check_dev("mask", mask, (B, L), (torch.uint8, torch.bool))
        if norm_weight is not None:
            _check_dev("norm_weight", norm_weight, (d,), (hidden.dtype,))
        mm = -1 if max_masked is None else int(max_masked)
        self.problem = make_problem(K, B, L, d, V, code, hidden, w_u, mask.view(torch.uint8), mm,
                                    norm_weight, norm_eps, norm_final)
        self.params = params.to_c()
        self.out = alloc_outputs(K, B, L, hidden.device, layer_stats)
        self.out_c = _outputs_struct(self.out)
        nbytes = int(lib().rpd_workspace_size(ctypes.byref(self.problem)))
        if nbytes == 0:
            raise ValueError("invalid problem shape")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=hidden.device)
        self._keep = (hidden, w_u, mask, norm_weight)

    def __call__(self, stream=None, events=None) -> dict:
        """Enqueue one call. ``events``: optional list of up to five
        ``torch.cuda.Event`` (or None) recorded at the stage boundaries
        (``rpd_score_commit_timed``)."""
        if events is None:
            _check(lib().rpd_score_commit(ctypes.byref(self.problem), ctypes.byref(self.params),
                                          ctypes.byref(self.out_c), self.workspace.data_ptr(),
                                          self.workspace.numel(), _stream_handle(stream)))
        else:
            arr = (ctypes.c_void_p * len(events))(*[None if e is None else e.cuda_event for e in events])
            _check(lib().rpd_score_commit_timed(ctypes.byref(self.problem), ctypes.byref(self.params),
                                                ctypes.byref(self.out_c), self.workspace.data_ptr(),
                                                self.workspace.numel(), _stream_handle(stream), arr,
                                                len(events)))
        return self.out


def score_commit(hidden: torch.Tensor, w_u: torch.Tensor, mask: torch.Tensor, params: Params,
                 max_masked: int | None = None, layer_stats: bool = False, stream=None,
                 norm_weight: torch.Tensor | None = None, norm_eps: float = 1e-5, norm_final: bool = False) -> dict:
    """``rpd_score_commit``: the whole commit step of one decoding iteration.

    hidden [K][B][L][d] and w_u [V][d] (bfloat16 or float32, same dtype,
    device, contiguous), mask [B][L] uint8/bool; optional norm_weight [d]
    (the gain of the model's final normalization, applied to layers 0..K-2,
    and to K-1 with norm_final). Returns the output tensors (see
    include/rpd.h), valid once the stream has run."""
    return ScoreCommit(hidden, w_u, mask, params, max_masked, layer_stats, norm_weight, norm_eps,
                       norm_final)(stream)


def gate_commit(mask: torch.Tensor, layer_argmax: torch.Tensor, layer_conf: torch.Tensor,
                layer_entropy: torch.Tensor, params: Params, stream=None) -> dict:
    """``rpd_gate_commit``: scoring and commitment from per-layer statistics
    ([K][B][L] int32 / float32 / float32 device tensors)."""
    K, B, L = layer_argmax.shape
    _check_dev("mask", mask, (B, L), (torch.uint8, torch.bool))
    _check_dev("layer_argmax", layer_argmax, (K, B, L), (torch.int32,))
    _check_dev("layer_conf", layer_conf, (K, B, L), (torch.float32,))
    _check_dev("layer_entropy", layer_entropy, (K, B, L), (torch.float32,))
    out = alloc_outputs(K, B, L, mask.device, False)
    oc = _outputs_struct(out)
    q = params.to_c()
    _check(lib().rpd_gate_commit(K, B, L, mask.view(torch.uint8).data_ptr(), layer_argmax.data_ptr(),
                                 layer_conf.data_ptr(), layer_entropy.data_ptr(), ctypes.byref(q),
                                 ctypes.byref(oc), _stream_handle(stream)))
    return out
