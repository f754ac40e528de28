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
ABI_VERSION = 3   # RPD_ABI_VERSION: the layouts and entry points this binding marshals for
PARAM_LAZY = 1
PARAM_LAZY_ALL = 2

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
    lazy_all: bool = False     # with lazy: every masked position walks its layers (RPD_PARAM_LAZY_ALL)

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
        flags = (PARAM_LAZY if self.lazy else 0) | (PARAM_LAZY_ALL if self.lazy_all else 0)
        return RpdParams(self.theta_h, self.theta_c, self.theta_s, self.w, int(self.k_max), self.beta,
                         int(self.window), flags, int(self.block), float(self.logit_scale))


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
        L.rpd_score_commit_noalloc.restype = ctypes.c_int
        L.rpd_score_commit_noalloc.argtypes = [ctypes.POINTER(RpdProblem), ctypes.POINTER(RpdParams),
                                               ctypes.POINTER(RpdOutputs), ctypes.c_void_p]
        L.rpd_gate_commit.restype = ctypes.c_int
        L.rpd_gate_commit.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.POINTER(RpdParams), ctypes.POINTER(RpdOutputs), ctypes.c_void_p]
        L.rpd_apply_commit.restype = ctypes.c_int
        L.rpd_apply_commit.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_void_p]
        L.rpd_status_string.restype = ctypes.c_char_p
        L.rpd_status_string.argtypes = [ctypes.c_int]
        L.rpd_last_error.restype = ctypes.c_char_p
        L.rpd_last_error.argtypes = []
        L.rpd_projection_variant.restype = ctypes.c_int32
        L.rpd_projection_variant.argtypes = [ctypes.POINTER(RpdProblem)]
        L.rpd_abi_version.restype = ctypes.c_int32
        L.rpd_abi_version.argtypes = []
        if L.rpd_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{_LIB_PATH} has ABI version {L.rpd_abi_version()}, this binding needs "
                               f"{ABI_VERSION}: rebuild the library")
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


PROJ_VARIANTS = {0: "bf16_s32", 1: "bf16_s64", 3: "f32", 4: "bf16_big", 6: "bf16_big192", 7: "bf16_big128"}


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


NOALLOC_SCRATCH_BYTES = 64 << 20   # RPD_NOALLOC_SCRATCH_BYTES


def score_commit_noalloc(hidden: torch.Tensor, w_u: torch.Tensor, mask: torch.Tensor, params: Params,
                         max_masked: int | None = None, layer_stats: bool = False, stream=None,
                         norm_weight: torch.Tensor | None = None, norm_eps: float = 1e-5, norm_final: bool = False,
                         out: dict | None = None) -> dict:
    """``rpd_score_commit_noalloc``: the commit step on the library's static
    scratch array instead of a workspace (for callers that cannot allocate
    device memory; calls that overlap on one GPU race). ``out``: output
    tensors from a previous call or ``alloc_outputs`` (allocated here if
    None). Returns the output tensors."""
    K, B, L, d = hidden.shape
    V = w_u.shape[0]
    _check_dev("hidden", hidden, (K, B, L, d), (hidden.dtype,))
    _check_dev("w_u", w_u, (V, d), (hidden.dtype,))
    _check_dev("mask", mask, (B, L), (torch.uint8, torch.bool))
    if norm_weight is not None:
        _check_dev("norm_weight", norm_weight, (d,), (hidden.dtype,))
    mm = -1 if max_masked is None else int(max_masked)
    problem = make_problem(K, B, L, d, V, _dtype_code(hidden), hidden, w_u, mask.view(torch.uint8), mm,
                           norm_weight, norm_eps, norm_final)
    o = alloc_outputs(K, B, L, hidden.device, layer_stats) if out is None else out
    q = params.to_c()
    oc = _outputs_struct(o)
    _check(lib().rpd_score_commit_noalloc(ctypes.byref(problem), ctypes.byref(q), ctypes.byref(oc),
                                          _stream_handle(stream)))
    return o


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


def apply_commit(mask: torch.Tensor, canvas: torch.Tensor, commit: torch.Tensor, token: torch.Tensor,
                 progress: torch.Tensor | None = None, step: torch.Tensor | None = None, stream=None) -> None:
    """``rpd_apply_commit``: committed positions take their token in the
    canvas and leave the mask (in place). mask [B][L] uint8/bool, canvas and
    token [B][L] int32, commit [B][L] uint8; optional progress int32
    [1 + n] (call counter, then the masked count left after each call) and
    step int32 [B][L] (the call index at which each position was filled)."""
    B, L = mask.shape
    _check_dev("mask", mask, (B, L), (torch.uint8, torch.bool))
    _check_dev("canvas", canvas, (B, L), (torch.int32,))
    _check_dev("commit", commit, (B, L), (torch.uint8,))
    _check_dev("token", token, (B, L), (torch.int32,))
    n = 0
    if progress is not None:
        if progress.dim() != 1 or progress.numel() < 1:
            raise ValueError("progress must be a 1-d tensor of at least one element")
        _check_dev("progress", progress, (progress.numel(),), (torch.int32,))
        n = progress.numel() - 1
    if step is not None:
        _check_dev("step", step, (B, L), (torch.int32,))
    _check(lib().rpd_apply_commit(B, L, mask.view(torch.uint8).data_ptr(), canvas.data_ptr(), commit.data_ptr(),
                                  token.data_ptr(), _ptr(progress), n, _ptr(step), _stream_handle(stream)))


class Decoder:
    """Iterations of the commit step until no position is masked (Section
    3.2): each iteration is ``rpd_score_commit`` followed by
    ``rpd_apply_commit`` on the same stream, over hidden states that stay
    fixed between iterations (they stand in for the forward passes of the
    model, which this library does not run).

    Every iteration commits at least one masked position (the progress
    fallback), so after t iterations at most n0 - t positions are masked; that
    bound is the ``max_masked`` of the call, and the masked count left after
    each iteration is recorded on the device (``progress``) and read back
    only every ``sync_every`` iterations, to tighten the bound and to stop.
    Iterations that find the canvas already full change nothing. With
    ``graph=True`` one iteration is captured in a HIP graph per plan and
    replayed: a plan is made for the first bound that needs it and serves
    every smaller bound of the same projection variant (down to half its
    bound for the variants whose grid grows with the rows). Plans are kept
    across ``reset()``, so repeated decodes replay the same graphs. A lazy
    call reads counts back while its bound exceeds 256 positions, so those
    iterations run eagerly and the rest replay graphs."""

    def __init__(self, hidden: torch.Tensor, w_u: torch.Tensor, mask: torch.Tensor, params: Params,
                 norm_weight: torch.Tensor | None = None, norm_eps: float = 1e-5, norm_final: bool = False,
                 graph: bool = True, sync_every: int = 8):
        K, B, L, d = hidden.shape
        _check_dev("mask", mask, (B, L), (torch.uint8, torch.bool))
        self.hidden, self.w_u, self.params = hidden, w_u, params
        self.norm = dict(norm_weight=norm_weight, norm_eps=norm_eps, norm_final=norm_final)
        self.sync_every = max(1, int(sync_every))
        self.shape = (K, B, L, d, w_u.shape[0])
        dev = hidden.device
        self.mask0 = mask.view(torch.uint8).clone()
        self.mask = self.mask0.clone()
        self.n0 = int(self.mask0.sum().item())
        self.graph = bool(graph)
        self.canvas = torch.full((B, L), -1, dtype=torch.int32, device=dev)
        self.step = torch.full((B, L), -1, dtype=torch.int32, device=dev)
        self.progress = torch.zeros(1 + max(self.n0, 1), dtype=torch.int32, device=dev)
        self._plans: dict[tuple, list] = {}   # (variant, captured) -> [(bound, ScoreCommit, graph or None)]
        self.captures = 0
        self.bounds: list[int] = []    # the max_masked of each enqueued iteration

    def reset(self) -> None:
        """Start a new decode from the initial mask (the plans are kept)."""
        self.mask.copy_(self.mask0)
        self.canvas.fill_(-1)
        self.step.fill_(-1)
        self.progress.zero_()
        self.bounds = []

    def _iteration(self, sc: ScoreCommit, events=None) -> None:
        o = sc(events=events)
        apply_commit(self.mask, self.canvas, o["commit"], o["token"], self.progress, self.step)

    def _plan_for(self, bound: int):
        K, B, L, d, V = self.shape
        variant = projection_variant(K, B, L, d, V, self.hidden.dtype, max_masked=bound)
        # a lazy call reads counts back (and cannot be captured) while its bound exceeds 256
        capture = self.graph and (not self.params.lazy or bound <= 256)
        plans = self._plans.setdefault((variant, capture), [])
        fits = [p for p in plans if p[0] >= bound and (variant.startswith("bf16_s") or 2 * bound > p[0])]
        if fits:
            return min(fits, key=lambda p: p[0])
        sc = ScoreCommit(self.hidden, self.w_u, self.mask, self.params, max_masked=bound, **self.norm)
        g = None
        if capture:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self._iteration(sc)
            self.captures += 1
        plans.append((bound, sc, g))
        return plans[-1]

    def run(self, max_iter: int | None = None, stage_events: bool = False) -> dict:
        """Decode until the canvas is full (or ``max_iter`` iterations);
        returns the canvas (-1 where never filled), the iteration at which
        each position was filled (``step``, -1 if never), the number of
        iterations that committed something (``iterations``, the NFE of the
        loop), the masked count left after each of them (``left``) and the
        number of enqueued iterations (``calls``). With ``stage_events``
        every iteration runs eagerly with events around its projection stage
        and ``proj_ms`` lists the projection time of each iteration."""
        limit = self.n0 if max_iter is None else min(int(max_iter), self.n0)
        t, known, t_known = 0, self.n0, 0
        ev = []
        while t < limit and known > 0:
            chunk = min(self.sync_every, limit - t)
            for _ in range(chunk):
                bound = max(known - (t - t_known), 1)
                bnd, sc, g = self._plan_for(bound)
                self.bounds.append(bnd)
                if stage_events:
                    pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for e in pair:         # torch creates the HIP event at its first record
                        e.record()
                    ev.append(pair)
                    self._iteration(sc, events=[None, pair[0], pair[1]])
                elif g is not None:
                    g.replay()
                else:
                    self._iteration(sc)
                t += 1
            known, t_known = int(self.progress[t].item()), t
        left = self.progress[1:1 + t].cpu().tolist()
        iters = next((i + 1 for i, n in enumerate(left) if n == 0), t)
        out = {"canvas": self.canvas, "step": self.step, "mask": self.mask, "iterations": iters,
               "left": left[:iters], "calls": t}
        if stage_events:
            torch.cuda.synchronize()
            out["proj_ms"] = [a.elapsed_time(b) for a, b in ev]
        return out
