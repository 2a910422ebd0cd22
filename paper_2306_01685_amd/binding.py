"""Thin ctypes binding of libmkor's C ABI (include/mkor.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels of libmkor.so.  PyTorch supplies device memory and streams.  There is
no fallback: if the library is missing or fails to load, every entry point
raises.

torch is imported before the library is loaded so that libmkor resolves to
the HIP runtime torch already loaded (one runtime per process; streams and
device pointers are shared).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch  # noqa: F401  (must precede loading libmkor, see module docstring)

_PKG = os.path.dirname(os.path.abspath(__file__))
# MKOR_LIBRARY selects another build of the same library (e.g. the
# sanitizer-instrumented one the host tests run against)
LIB_PATH = os.environ.get("MKOR_LIBRARY") or os.path.join(_PKG, "libmkor.so")

MKOR_OK = 0
MKOR_INVALID_ARG = -1
MKOR_WORKSPACE_TOO_SMALL = -2
MKOR_UNSUPPORTED = -3
MKOR_HIP_ERROR = -4

SM_EXACT = 0
SM_PAPER_EQ6 = 1
NORM_INF = 0
NORM_MAXABS = 1
DTYPE_F32 = 0
DTYPE_BF16 = 1
MAX_DIM = 32768
MAX_ROWS = 1 << 26
MAX_RANK = 4
ABI_VERSION = 10
NOALLOC_MAX_BYTES = 64 << 20
GEMM_AUTO = 0
GEMM_FP32 = 1
GEMM_SPLIT = 2
GEMM_PATHS = {"auto": GEMM_AUTO, "fp32": GEMM_FP32, "split": GEMM_SPLIT}
OPT_SGD = 1
OPT_LAMB = 2


class mkor_params(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_float), ("zeta", ctypes.c_float), ("stab_eps", ctypes.c_float),
                ("norm_kind", ctypes.c_int32), ("sm_variant", ctypes.c_int32),
                ("rescale", ctypes.c_int32), ("guard_nonfinite", ctypes.c_int32)]


class mkor_layer(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("second_order", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("Linv", ctypes.c_void_p), ("Rinv", ctypes.c_void_p),
                ("a", ctypes.c_void_p), ("g", ctypes.c_void_p),
                ("G", ctypes.c_void_p), ("dW", ctypes.c_void_p), ("stats", ctypes.c_void_p),
                ("rows", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("A", ctypes.c_void_p), ("Gout", ctypes.c_void_p),
                ("factor_dtype", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("W", ctypes.c_void_p), ("opt_m", ctypes.c_void_p), ("opt_v", ctypes.c_void_p),
                ("gemm_path", ctypes.c_int32), ("reserved0", ctypes.c_int32)]


class mkor_opt_params(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("step", ctypes.c_int32), ("lr", ctypes.c_float),
                ("momentum", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float), ("store_dw", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class mkor_layer_stats(ctypes.Structure):
    _fields_ = [("nu_L", ctypes.c_float), ("nu_R", ctypes.c_float),
                ("s_L", ctypes.c_float), ("s_R", ctypes.c_float),
                ("norm_G", ctypes.c_float), ("norm_dW_hat", ctypes.c_float), ("scale", ctypes.c_float),
                ("stab_L", ctypes.c_int32), ("stab_R", ctypes.c_int32),
                ("skip_L", ctypes.c_int32), ("skip_R", ctypes.c_int32),
                ("nonfinite_scale", ctypes.c_int32)]


class mkor_hybrid_params(ctypes.Structure):
    _fields_ = [("window", ctypes.c_int32), ("patience", ctypes.c_int32), ("warmup", ctypes.c_int32),
                ("threshold", ctypes.c_float)]


class mkor_hybrid_state(ctypes.Structure):
    _fields_ = [("params", mkor_hybrid_params), ("sum", ctypes.c_double), ("prev_mean", ctypes.c_double),
                ("last_rate", ctypes.c_double), ("observed", ctypes.c_int64), ("switched_at", ctypes.c_int64),
                ("count", ctypes.c_int32), ("windows", ctypes.c_int32), ("slow", ctypes.c_int32),
                ("second_order", ctypes.c_int32)]


STATS_BYTES = ctypes.sizeof(mkor_layer_stats)
STATS_FIELDS = [f for f, _ in mkor_layer_stats._fields_]

EXPORTED = ["mkor_abi_version", "mkor_status_string", "mkor_last_error", "mkor_params_check",
            "mkor_workspace_size", "mkor_plan_create", "mkor_update_factors",
            "mkor_precondition", "mkor_step", "mkor_run_stage", "mkor_sync_factors",
            "mkor_opt_params_check", "mkor_step_opt", "mkor_precondition_opt", "mkor_step_noalloc",
            "mkor_set_second_order", "mkor_factors_pending", "mkor_hybrid_init", "mkor_hybrid_observe",
            "mkor_plan_destroy"]

# MKOR_STAGE_*, in launch order
STAGE_NAMES = ["means", "sm_pass", "sm_finalize", "gemm_prep", "gemm_xt", "gemm_dw", "rescale"]
(STAGE_MEANS, STAGE_SM_PASS, STAGE_SM_FINALIZE, STAGE_GEMM_PREP, STAGE_GEMM_XT, STAGE_GEMM_DW,
 STAGE_RESCALE) = range(len(STAGE_NAMES))
NUM_STAGES = len(STAGE_NAMES)


class MkorError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {status_string(status)} ({status}): {detail}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libmkor.so once; raises if it is absent (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libmkor.so not found at {path}: build it with "
                           "`python -m paper_2306_01685_amd.build` (or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.mkor_abi_version.restype = ctypes.c_int
    lib.mkor_abi_version.argtypes = []
    lib.mkor_status_string.restype = ctypes.c_char_p
    lib.mkor_status_string.argtypes = [ctypes.c_int]
    lib.mkor_last_error.restype = ctypes.c_char_p
    lib.mkor_last_error.argtypes = []
    lib.mkor_params_check.restype = ctypes.c_int
    lib.mkor_params_check.argtypes = [ctypes.POINTER(mkor_params)]
    lib.mkor_workspace_size.restype = ctypes.c_int
    lib.mkor_workspace_size.argtypes = [ctypes.POINTER(mkor_layer), I32, ctypes.POINTER(SZ)]
    lib.mkor_plan_create.restype = ctypes.c_int
    lib.mkor_plan_create.argtypes = [ctypes.POINTER(mkor_layer), I32, P, SZ, ctypes.POINTER(P)]
    for name in ("mkor_update_factors", "mkor_precondition", "mkor_step"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [P, ctypes.POINTER(mkor_params), P]
    lib.mkor_run_stage.restype = ctypes.c_int
    lib.mkor_run_stage.argtypes = [P, ctypes.POINTER(mkor_params), I32, P]
    lib.mkor_sync_factors.restype = ctypes.c_int
    lib.mkor_sync_factors.argtypes = [P, P]
    lib.mkor_opt_params_check.restype = ctypes.c_int
    lib.mkor_opt_params_check.argtypes = [ctypes.POINTER(mkor_opt_params)]
    for name in ("mkor_step_opt", "mkor_precondition_opt"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [P, ctypes.POINTER(mkor_params), ctypes.POINTER(mkor_opt_params), P]
    lib.mkor_step_noalloc.restype = ctypes.c_int
    lib.mkor_step_noalloc.argtypes = [ctypes.POINTER(mkor_layer), I32, ctypes.POINTER(mkor_params), P]
    lib.mkor_set_second_order.restype = ctypes.c_int
    lib.mkor_set_second_order.argtypes = [P, ctypes.POINTER(I32), P]
    lib.mkor_factors_pending.restype = ctypes.c_int
    lib.mkor_factors_pending.argtypes = [P, ctypes.POINTER(I32)]
    lib.mkor_hybrid_init.restype = ctypes.c_int
    lib.mkor_hybrid_init.argtypes = [ctypes.POINTER(mkor_hybrid_params), ctypes.POINTER(mkor_hybrid_state)]
    lib.mkor_hybrid_observe.restype = ctypes.c_int
    lib.mkor_hybrid_observe.argtypes = [ctypes.POINTER(mkor_hybrid_state), ctypes.c_float, ctypes.POINTER(I32)]
    lib.mkor_plan_destroy.restype = None
    lib.mkor_plan_destroy.argtypes = [P]
    if lib.mkor_abi_version() != ABI_VERSION:
        raise RuntimeError(f"libmkor ABI {lib.mkor_abi_version()} != binding ABI {ABI_VERSION}")
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().mkor_status_string(status).decode()


def last_error() -> str:
    return load_library().mkor_last_error().decode()


def _check(status: int, where: str):
    if status != MKOR_OK:
        raise MkorError(status, where, last_error())


@dataclass
class Params:
    gamma: float = 0.9
    zeta: float = 0.5
    eps: float = 100.0
    norm_kind: int = NORM_INF
    variant: int = SM_EXACT
    rescale: bool = True
    guard_nonfinite: bool = True

    def to_c(self) -> mkor_params:
        return mkor_params(self.gamma, self.zeta, self.eps,
                           int(self.norm_kind), int(self.variant), int(bool(self.rescale)),
                           int(bool(self.guard_nonfinite)))


@dataclass
class OptParams:
    """Backend optimizer fused with the rescale (mkor_opt_params)."""
    kind: int = OPT_LAMB
    step: int = 1
    lr: float = 1e-3
    momentum: float = 0.9
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-6
    weight_decay: float = 0.01
    store_dw: bool = False

    def to_c(self) -> mkor_opt_params:
        return mkor_opt_params(int(self.kind), int(self.step), self.lr, self.momentum, self.beta1,
                               self.beta2, self.eps, self.weight_decay, int(bool(self.store_dw)), 0)


def opt_params_check(o) -> int:
    c = o.to_c() if isinstance(o, OptParams) else o
    return load_library().mkor_opt_params_check(ctypes.byref(c))


def params_check(p) -> int:
    c = p.to_c() if isinstance(p, Params) else p
    return load_library().mkor_params_check(ctypes.byref(c))


def make_layer_array(descs):
    """descs: list of dicts with integer fields and raw pointer values."""
    arr = (mkor_layer * max(1, len(descs)))()
    for i, d in enumerate(descs):
        arr[i] = mkor_layer(d["d_in"], d["d_out"], d.get("second_order", 1), d.get("grad_dtype", 0),
                            d.get("Linv") or None, d.get("Rinv") or None, d.get("a") or None,
                            d.get("g") or None, d.get("G") or None, d.get("dW") or None,
                            d.get("stats") or None, d.get("rows", 0), d.get("act_dtype", 0),
                            d.get("A") or None, d.get("Gout") or None, d.get("factor_dtype", 0),
                            d.get("rank", 0), d.get("W") or None, d.get("opt_m") or None,
                            d.get("opt_v") or None, d.get("gemm_path", 0), d.get("reserved0", 0))
    return arr


def workspace_size_raw(descs) -> int:
    arr = make_layer_array(descs)
    out = ctypes.c_size_t(0)
    _check(load_library().mkor_workspace_size(arr, len(descs), ctypes.byref(out)), "mkor_workspace_size")
    return out.value


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream_handle(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def layer_descs(layers):
    """mkor_layer field values (raw device pointers) of a list of layer dicts
    holding torch tensors (see MkorPlan)."""
    descs = []
    for L in layers:
        so = int(bool(L.get("second_order", True)))
        G = L["G"]
        if G.dtype == torch.bfloat16:
            gdt = DTYPE_BF16
        elif G.dtype == torch.float32:
            gdt = DTYPE_F32
        else:
            raise TypeError(f"unsupported gradient dtype {G.dtype}")
        for k in ("Linv", "Rinv", "a", "g", "G", "dW", "A", "Gout", "W", "opt_m", "opt_v"):
            t = L.get(k)
            if t is not None and not t.is_contiguous():
                raise ValueError(f"{k} must be contiguous")
        fdt = DTYPE_F32
        if so:
            dts = {L["Linv"].dtype, L["Rinv"].dtype}
            if dts == {torch.bfloat16}:
                fdt = DTYPE_BF16
            elif dts != {torch.float32}:
                raise TypeError("Linv and Rinv must both be fp32 or both bf16")
        A = L.get("A")
        rows, adt = 0, DTYPE_F32
        if A is not None:
            rows = int(A.shape[0])
            adt = DTYPE_BF16 if A.dtype == torch.bfloat16 else DTYPE_F32
            if A.dtype not in (torch.bfloat16, torch.float32) or L["Gout"].dtype != A.dtype:
                raise TypeError("A and Gout must both be fp32 or both bf16")
        descs.append(dict(d_in=int(L["d_in"]), d_out=int(L["d_out"]), second_order=so,
                          grad_dtype=gdt, Linv=_ptr(L.get("Linv")), Rinv=_ptr(L.get("Rinv")),
                          a=_ptr(L.get("a")), g=_ptr(L.get("g")), G=_ptr(G), dW=_ptr(L["dW"]),
                          stats=_ptr(L.get("stats")), rows=rows, act_dtype=adt, A=_ptr(A),
                          Gout=_ptr(L.get("Gout")), factor_dtype=fdt,
                          rank=int(L["a"].shape[0]) if so and L["a"].dim() == 2 else 0,
                          W=_ptr(L.get("W")), opt_m=_ptr(L.get("opt_m")), opt_v=_ptr(L.get("opt_v")),
                          gemm_path=GEMM_PATHS[L.get("gemm_path", "auto")]))
    return descs


class MkorPlan:
    """A plan over a grouped list of layers, holding torch device tensors.

    Each layer is a dict with d_in, d_out and tensors Linv, Rinv (symmetric;
    both fp32, or both bf16 for half-precision factors), a, g (fp32 vectors of
    length d_in / d_out, or (r, d_in) / (r, d_out) arrays of r vectors for a
    rank-r update), G (fp32 or bf16, d_in x d_out), dW (fp32, d_in x d_out),
    optional second_order (default True), optional stats
    (a uint8 device tensor of STATS_BYTES bytes), and optionally token rows A
    (rows x d_in) and Gout (rows x d_out), fp32 or bf16, from which each step
    forms a and g (their means), and optionally gemm_path ("auto", "fp32" or
    "split": how the preconditioning of fp32 factors multiplies; default
    "auto").  The plan owns its workspace
    (a torch uint8 tensor) and keeps references to every tensor it was given.

    After step() / update_factors() the Linv / Rinv tensors lag the current
    factors by one pending rank-1 term held in the workspace; sync_factors()
    writes the current factors into them (include/mkor.h, "Factor state").
    """

    def __init__(self, layers, device=None, workspace=None):
        self._lib = load_library()
        self.layers = layers
        descs = layer_descs(layers)
        self._arr = make_layer_array(descs)
        n = len(descs)
        size = ctypes.c_size_t(0)
        _check(self._lib.mkor_workspace_size(self._arr, n, ctypes.byref(size)), "mkor_workspace_size")
        self.ws_bytes = size.value
        if workspace is not None:
            # the caller's workspace: a uint8 device tensor of at least ws_bytes,
            # 256-byte aligned (checked by mkor_plan_create)
            if workspace.dtype != torch.uint8 or not workspace.is_contiguous():
                raise TypeError("workspace must be a contiguous uint8 tensor")
            self._ws_raw = workspace
            self.workspace = workspace
            base, off = workspace.data_ptr(), 0
            ws_len = workspace.numel()
        else:
            if device is None:
                device = layers[0]["dW"].device if layers else torch.device("cuda")
            # over-allocate by 256 bytes and align the base to 256
            self._ws_raw = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
            base = self._ws_raw.data_ptr()
            off = (-base) % 256
            self.workspace = self._ws_raw[off:off + self.ws_bytes]
            ws_len = self.ws_bytes
        plan = ctypes.c_void_p(None)
        _check(self._lib.mkor_plan_create(self._arr, n, ctypes.c_void_p(base + off), ws_len,
                                          ctypes.byref(plan)), "mkor_plan_create")
        self._plan = plan

    def _call(self, name, params, stream):
        p = params.to_c() if isinstance(params, Params) else params
        fn = getattr(self._lib, name)
        _check(fn(self._plan, ctypes.byref(p), _stream_handle(stream)), name)

    def update_factors(self, params: Params, stream=None):
        self._call("mkor_update_factors", params, stream)

    def precondition(self, params: Params, stream=None):
        self._call("mkor_precondition", params, stream)

    def step(self, params: Params, stream=None):
        self._call("mkor_step", params, stream)

    def run_stage(self, params: Params, stage: int, stream=None):
        p = params.to_c() if isinstance(params, Params) else params
        _check(self._lib.mkor_run_stage(self._plan, ctypes.byref(p), int(stage), _stream_handle(stream)),
               "mkor_run_stage")

    def step_opt(self, params: Params, opt: "OptParams", stream=None):
        """mkor_step with the backend optimizer fused into the rescale."""
        p, o = params.to_c(), opt.to_c()
        _check(self._lib.mkor_step_opt(self._plan, ctypes.byref(p), ctypes.byref(o), _stream_handle(stream)),
               "mkor_step_opt")

    def precondition_opt(self, params: Params, opt: "OptParams", stream=None):
        p, o = params.to_c(), opt.to_c()
        _check(self._lib.mkor_precondition_opt(self._plan, ctypes.byref(p), ctypes.byref(o),
                                               _stream_handle(stream)), "mkor_precondition_opt")

    def sync_factors(self, stream=None):
        _check(self._lib.mkor_sync_factors(self._plan, _stream_handle(stream)), "mkor_sync_factors")

    def set_second_order(self, flags, stream=None):
        """MKOR-H: the branch of each layer for the following calls (1
        second-order, 0 first-order), one entry per layer of the plan."""
        n = len(self.layers)
        if len(flags) != n:
            raise ValueError(f"{len(flags)} flags for {n} layers")
        arr = (ctypes.c_int32 * max(1, n))(*[int(f) for f in flags])
        _check(self._lib.mkor_set_second_order(self._plan, arr, _stream_handle(stream)), "mkor_set_second_order")

    def factors_pending(self) -> bool:
        """True when Linv / Rinv may lag the current factors (sync_factors needed)."""
        out = ctypes.c_int32(0)
        _check(self._lib.mkor_factors_pending(self._plan, ctypes.byref(out)), "mkor_factors_pending")
        return bool(out.value)

    def close(self):
        if getattr(self, "_plan", None) is not None and self._plan.value:
            self._lib.mkor_plan_destroy(self._plan)
            self._plan = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Hybrid:
    """MKOR-H's switching rule (mkor_hybrid_init / mkor_hybrid_observe): feed
    one loss per iteration; `second_order` turns False once the windowed loss
    decrease has stayed below `threshold` for `patience` windows."""

    def __init__(self, window=10, patience=2, warmup=1, threshold=0.01):
        self._lib = load_library()
        self.params = mkor_hybrid_params(int(window), int(patience), int(warmup), float(threshold))
        self.state = mkor_hybrid_state()
        _check(self._lib.mkor_hybrid_init(ctypes.byref(self.params), ctypes.byref(self.state)), "mkor_hybrid_init")

    def observe(self, loss: float) -> bool:
        out = ctypes.c_int32(1)
        _check(self._lib.mkor_hybrid_observe(ctypes.byref(self.state), float(loss), ctypes.byref(out)),
               "mkor_hybrid_observe")
        return bool(out.value)

    @property
    def second_order(self) -> bool:
        return bool(self.state.second_order)

    @property
    def switched_at(self):
        return None if self.state.switched_at < 0 else int(self.state.switched_at)


def step_noalloc(layers, params: Params, stream=None):
    """One full step over `layers` (dicts of torch tensors, as for MkorPlan)
    through mkor_step_noalloc: no workspace, no device allocation; the
    factors are updated in place."""
    descs = layer_descs(layers)
    arr = make_layer_array(descs)
    p = params.to_c() if isinstance(params, Params) else params
    _check(load_library().mkor_step_noalloc(arr, len(descs), ctypes.byref(p), _stream_handle(stream)),
           "mkor_step_noalloc")


def read_stats(stats_tensor) -> dict:
    """Decodes one mkor_layer_stats record from a uint8 tensor (any device)."""
    raw = bytes(stats_tensor.detach().cpu().numpy().tobytes())
    s = mkor_layer_stats.from_buffer_copy(raw[:STATS_BYTES])
    return {f: getattr(s, f) for f in STATS_FIELDS}
