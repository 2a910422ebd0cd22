"""C ABI host-side behaviour, without a GPU.

Every validation path of include/mkor.h returns its status before the first
HIP call, so these tests pass fake (never dereferenced) device addresses.
"""
import ctypes
import math
import os
import re

import pytest

import paper_2306_01685_amd as M
from paper_2306_01685_amd import binding as B
from tests.test_rank1_gpu import INTERMEDIATE   # plans at 1024 / 2048 / 4096 rows per block

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(M.LIB_PATH):
        pytest.fail("libmkor.so is not built (run python -m paper_2306_01685_amd.build)")
    return M.load_library()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "mkor.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mkor_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(M.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n
    assert lib.mkor_abi_version() == M.binding.ABI_VERSION


def test_status_strings(lib):
    for code, name in [(0, "MKOR_OK"), (-1, "MKOR_INVALID_ARG"), (-2, "MKOR_WORKSPACE_TOO_SMALL"),
                       (-3, "MKOR_UNSUPPORTED"), (-4, "MKOR_HIP_ERROR")]:
        assert M.status_string(code) == name
    assert M.status_string(7) == "MKOR_UNKNOWN_STATUS"


def test_struct_sizes():
    assert ctypes.sizeof(B.mkor_params) == 28
    assert ctypes.sizeof(B.mkor_layer) == 16 + 7 * 8 + 8 + 2 * 8 + 8 + 3 * 8 + 8
    assert ctypes.sizeof(B.mkor_opt_params) == 40
    assert M.STATS_BYTES == 48


@pytest.mark.parametrize("field,value", [
    ("gamma", 0.0), ("gamma", 1.0), ("gamma", math.nan), ("gamma", -0.5),
    ("zeta", 0.0), ("zeta", 1.5), ("zeta", math.nan),
    ("eps", math.nan), ("eps", -1.0),
    ("norm_kind", 2), ("variant", 7), ("rescale", 2), ("guard_nonfinite", 3),
])
def test_params_rejected(lib, field, value):
    p = M.Params()
    setattr(p, field, value)
    c = p.to_c()
    if field in ("rescale", "guard_nonfinite"):
        setattr(c, field, value)
    assert M.params_check(c) == M.MKOR_INVALID_ARG
    assert M.last_error()


@pytest.mark.parametrize("kw", [dict(), dict(eps=math.inf), dict(eps=0.0), dict(zeta=1.0),
                                dict(variant=1, norm_kind=1, rescale=False, guard_nonfinite=False)])
def test_params_accepted(lib, kw):
    assert M.params_check(M.Params(**kw)) == M.MKOR_OK


def test_params_null(lib):
    assert lib.mkor_params_check(None) == M.MKOR_INVALID_ARG


# ------------------------------------------------------------------ fake address space

class Fake:
    """Hands out disjoint, 256-byte aligned fake device addresses."""

    def __init__(self):
        self.next = 0x7F0000000000

    def alloc(self, nbytes):
        p = self.next
        self.next += (nbytes + 4095) // 4096 * 4096 + 4096
        return p


def layer(fk, d_in, d_out, so=1, dt=0, stats=False, rows=0, adt=0, fdt=0, rank=0):
    esz = 2 if dt == 1 else 4
    aesz = 2 if adt == 1 else 4
    fsz = 2 if fdt == 1 else 4
    return dict(d_in=d_in, d_out=d_out, second_order=so, grad_dtype=dt, factor_dtype=fdt,
                Linv=fk.alloc(d_in * d_in * fsz), Rinv=fk.alloc(d_out * d_out * fsz),
                a=fk.alloc(d_in * 4 * max(1, rank)), g=fk.alloc(d_out * 4 * max(1, rank)),
                G=fk.alloc(d_in * d_out * esz), rank=rank,
                dW=fk.alloc(d_in * d_out * 4), stats=fk.alloc(48) if stats else None,
                rows=rows, act_dtype=adt,
                A=fk.alloc(rows * d_in * aesz) if rows else None,
                Gout=fk.alloc(rows * d_out * aesz) if rows else None)


def ws_status(descs):
    arr = B.make_layer_array(descs)
    out = ctypes.c_size_t(0)
    st = M.load_library().mkor_workspace_size(arr, len(descs), ctypes.byref(out))
    return st, out.value


def test_workspace_size_covers_intermediate(lib):
    fk = Fake()
    descs = [layer(fk, 1024, 4096, dt=1), layer(fk, 4096, 1024), layer(fk, 37, 100, so=0)]
    st, size = ws_status(descs)
    assert st == M.MKOR_OK
    # X = Linv G is kept per second-order layer (fp32), plus tables and vectors
    assert size >= 4 * (1024 * 4096 * 2)
    assert size < 4 * (1024 * 4096 * 2) + (8 << 20)
    assert size % 256 == 0


def test_empty_list(lib):
    st, size = ws_status([])
    assert st == M.MKOR_OK and size == 0
    plan = ctypes.c_void_p(None)
    assert lib.mkor_plan_create(None, 0, None, 0, ctypes.byref(plan)) == M.MKOR_OK
    p = M.Params().to_c()
    for fn in (lib.mkor_update_factors, lib.mkor_precondition, lib.mkor_step):
        assert fn(plan, ctypes.byref(p), None) == M.MKOR_OK
    assert lib.mkor_sync_factors(plan, None) == M.MKOR_OK
    lib.mkor_plan_destroy(plan)
    lib.mkor_plan_destroy(None)


@pytest.mark.parametrize("mutate,status", [
    (lambda L: L.update(d_in=0), M.MKOR_INVALID_ARG),
    (lambda L: L.update(d_out=M.MAX_DIM + 1), M.MKOR_INVALID_ARG),
    (lambda L: L.update(second_order=2), M.MKOR_INVALID_ARG),
    (lambda L: L.update(grad_dtype=5), M.MKOR_UNSUPPORTED),
    (lambda L: L.update(G=None), M.MKOR_INVALID_ARG),
    (lambda L: L.update(dW=None), M.MKOR_INVALID_ARG),
    (lambda L: L.update(Linv=None), M.MKOR_INVALID_ARG),
    (lambda L: L.update(g=None), M.MKOR_INVALID_ARG),
    (lambda L: L.update(a=L["a"] + 4), M.MKOR_INVALID_ARG),        # misaligned
    (lambda L: L.update(dW=L["G"]), M.MKOR_INVALID_ARG),           # output aliases input
    (lambda L: L.update(Rinv=L["Linv"] + 256), M.MKOR_INVALID_ARG),  # factors overlap
    (lambda L: L.update(stats=L["dW"] + 64), M.MKOR_INVALID_ARG),  # stats inside dW
    (lambda L: L.update(rows=-1), M.MKOR_INVALID_ARG),
    (lambda L: L.update(rows=M.MAX_ROWS + 1), M.MKOR_INVALID_ARG),
    (lambda L: L.update(rows=8), M.MKOR_INVALID_ARG),              # rows > 0 without A / Gout
    (lambda L: L.update(factor_dtype=2), M.MKOR_UNSUPPORTED),
    (lambda L: L.update(rank=-1), M.MKOR_INVALID_ARG),
    (lambda L: L.update(rank=5), M.MKOR_INVALID_ARG),
    (lambda L: L.update(factor_dtype=1, d_out=100), M.MKOR_UNSUPPORTED),  # bf16: multiples of 64
])
def test_layer_rejected(lib, mutate, status):
    fk = Fake()
    descs = [layer(fk, 64, 96), layer(fk, 40, 40)]
    mutate(descs[0])
    st, _ = ws_status(descs)
    assert st == status, M.last_error()
    assert M.last_error()


def test_cross_layer_aliasing(lib):
    fk = Fake()
    a, b = layer(fk, 64, 64), layer(fk, 64, 64)
    b["dW"] = a["dW"]                      # two outputs on one buffer
    assert ws_status([a, b])[0] == M.MKOR_INVALID_ARG
    a, b = layer(fk, 64, 64), layer(fk, 64, 64)
    b["Linv"] = a["G"]                     # factor written over another layer's input
    assert ws_status([a, b])[0] == M.MKOR_INVALID_ARG
    a, b = layer(fk, 64, 64), layer(fk, 64, 64)
    b["a"] = a["a"]                        # read-only inputs may be shared
    b["G"] = a["G"]
    assert ws_status([a, b])[0] == M.MKOR_OK


def test_rank1_rows_validation(lib):
    fk = Fake()
    L = layer(fk, 64, 96, rows=128, adt=1)
    assert ws_status([L])[0] == M.MKOR_OK
    L = layer(fk, 64, 96, rows=128, adt=1)
    L["act_dtype"] = 7
    assert ws_status([L])[0] == M.MKOR_UNSUPPORTED
    L = layer(fk, 64, 96, rows=128)
    L["A"] += 8                                  # misaligned
    assert ws_status([L])[0] == M.MKOR_INVALID_ARG
    L = layer(fk, 64, 96, rows=128)
    L["Gout"] = L["A"]                           # inputs may be shared (read-only)
    assert ws_status([L])[0] == M.MKOR_OK
    L = layer(fk, 64, 96, rows=128)
    L["a"] = L["A"]                              # written mean over an input
    assert ws_status([L])[0] == M.MKOR_INVALID_ARG
    a, b = layer(fk, 64, 64), layer(fk, 64, 64, rows=16)
    b["a"] = a["a"]                              # a is written for b: no sharing
    assert ws_status([a, b])[0] == M.MKOR_INVALID_ARG
    L = layer(fk, 64, 96, so=0, rows=16)
    assert ws_status([L])[0] == M.MKOR_INVALID_ARG   # rows only for second-order layers


def test_workspace_grows_with_rows(lib):
    fk = Fake()
    base = ws_status([layer(fk, 1024, 4096)])[1]
    with_rows = ws_status([layer(fk, 1024, 4096, rows=16384, adt=1)])[1]
    # float64 partial sums: (1024 + 4096) / 512 chunks x 32 row blocks x 512 (one
    # layer gives too few blocks for more than the smallest, 512 rows per block)
    assert with_rows - base >= 8 * (1024 + 4096) * 32
    assert with_rows - base < 8 * (1024 + 4096) * 32 + (1 << 20)


@pytest.mark.parametrize("n,shape,rows,rpb", [(1, (1024, 4096), 16384, 512)] + INTERMEDIATE)
def test_mean_rows_per_block_rule(lib, n, shape, rows, rpb):
    """The plan's rows per block of the column-mean partials, seen through the
    workspace size: the partials of the expected block size fit in what the
    rows add, those of half that size (about twice as many) do not."""
    fk = Fake()
    base = ws_status([layer(fk, *shape) for _ in range(n)])[1]
    extra = ws_status([layer(fk, *shape, rows=rows, adt=1) for _ in range(n)])[1] - base

    def partials(r):
        return 8 * 512 * n * (-(-shape[0] // 512) + -(-shape[1] // 512)) * -(-rows // r)
    assert partials(rpb) <= extra < partials(rpb // 2)


def test_first_order_layer_needs_no_factors(lib):
    fk = Fake()
    L = layer(fk, 50, 70, so=0)
    L.update(Linv=None, Rinv=None, a=None, g=None)
    assert ws_status([L])[0] == M.MKOR_OK


def test_plan_create_workspace_errors(lib):
    fk = Fake()
    descs = [layer(fk, 64, 96)]
    st, size = ws_status(descs)
    arr = B.make_layer_array(descs)
    plan = ctypes.c_void_p(None)
    ws = fk.alloc(size + 4096)
    assert lib.mkor_plan_create(arr, 1, ws, size - 256, ctypes.byref(plan)) == M.MKOR_WORKSPACE_TOO_SMALL
    assert lib.mkor_plan_create(arr, 1, None, size, ctypes.byref(plan)) == M.MKOR_INVALID_ARG
    assert lib.mkor_plan_create(arr, 1, ws + 16, size, ctypes.byref(plan)) == M.MKOR_INVALID_ARG
    assert lib.mkor_plan_create(arr, 1, ws, size, None) == M.MKOR_INVALID_ARG
    # workspace overlapping a layer buffer
    assert lib.mkor_plan_create(arr, 1, descs[0]["dW"] // 256 * 256, size,
                                ctypes.byref(plan)) == M.MKOR_INVALID_ARG
    assert lib.mkor_plan_create(arr, -1, ws, size, ctypes.byref(plan)) == M.MKOR_INVALID_ARG
    assert not plan.value


def test_entry_points_reject_before_device(lib):
    p = M.Params().to_c()
    for fn in (lib.mkor_update_factors, lib.mkor_precondition, lib.mkor_step):
        assert fn(None, ctypes.byref(p), None) == M.MKOR_INVALID_ARG
    assert lib.mkor_sync_factors(None, None) == M.MKOR_INVALID_ARG
    assert lib.mkor_run_stage(None, ctypes.byref(p), 0, None) == M.MKOR_INVALID_ARG
    plan = ctypes.c_void_p(None)
    assert lib.mkor_plan_create(None, 0, None, 0, ctypes.byref(plan)) == M.MKOR_OK
    bad = M.Params(gamma=2.0).to_c()
    for fn in (lib.mkor_update_factors, lib.mkor_precondition, lib.mkor_step):
        assert fn(plan, ctypes.byref(bad), None) == M.MKOR_INVALID_ARG
        assert fn(plan, None, None) == M.MKOR_INVALID_ARG
    for stage in (-1, M.NUM_STAGES):
        assert lib.mkor_run_stage(plan, ctypes.byref(p), stage, None) == M.MKOR_INVALID_ARG
    lib.mkor_plan_destroy(plan)


def test_bf16_factor_layers(lib):
    fk = Fake()
    # bf16 factors: d_in, d_out multiples of 64, factor buffers 2 bytes/element
    assert ws_status([layer(fk, 64, 192, fdt=1)])[0] == M.MKOR_OK
    assert ws_status([layer(fk, 64, 96, fdt=1)])[0] == M.MKOR_UNSUPPORTED
    # a first-order layer ignores factor_dtype's shape rule
    assert ws_status([layer(fk, 50, 70, so=0, fdt=1)])[0] == M.MKOR_OK
    # the bf16 factor of one layer may sit right after the other (2-byte extent)
    L = layer(fk, 128, 128, fdt=1)
    L["Rinv"] = L["Linv"] + 128 * 128 * 2
    assert ws_status([L])[0] == M.MKOR_OK
    L["Rinv"] = L["Linv"] + 128 * 128 * 2 - 256
    assert ws_status([L])[0] == M.MKOR_INVALID_ARG


def test_workspace_bf16_factors(lib):
    fk = Fake()
    f32 = ws_status([layer(fk, 1024, 4096, dt=1)])[1]
    h = ws_status([layer(fk, 1024, 4096, dt=1, fdt=1)])[1]
    # the intermediate (X^T fp32, or Y^T bf16) is d_in x d_out
    assert f32 - h >= 2 * 1024 * 4096 - (1 << 20)
    assert h >= 2 * 1024 * 4096
    # an fp32 gradient of a bf16-factor layer also gets a bf16 copy
    h32 = ws_status([layer(fk, 1024, 4096, fdt=1)])[1]
    assert h32 - h >= 2 * 1024 * 4096
    # mixed lists plan both GEMM kinds
    st, _ = ws_status([layer(fk, 1024, 4096, fdt=1), layer(fk, 4096, 1024), layer(fk, 37, 100)])
    assert st == M.MKOR_OK


def test_gemm_path_validation(lib):
    fk = Fake()
    for path in (M.GEMM_AUTO, M.GEMM_FP32, M.GEMM_SPLIT):
        assert ws_status([dict(layer(fk, 64, 128), gemm_path=path)])[0] == M.MKOR_OK
    for path in (-1, 3):
        assert ws_status([dict(layer(fk, 64, 128), gemm_path=path)])[0] == M.MKOR_INVALID_ARG
    # the split needs multiples of 64; AUTO and FP32 take any shape
    assert ws_status([dict(layer(fk, 64, 96), gemm_path=M.GEMM_SPLIT)])[0] == M.MKOR_UNSUPPORTED
    assert ws_status([dict(layer(fk, 37, 100), gemm_path=M.GEMM_AUTO)])[0] == M.MKOR_OK
    assert ws_status([dict(layer(fk, 37, 100), gemm_path=M.GEMM_FP32)])[0] == M.MKOR_OK
    # only for second-order layers with fp32 factors
    assert ws_status([dict(layer(fk, 64, 128, fdt=1), gemm_path=M.GEMM_SPLIT)])[0] == M.MKOR_INVALID_ARG
    assert ws_status([dict(layer(fk, 64, 128, so=0), gemm_path=M.GEMM_FP32)])[0] == M.MKOR_INVALID_ARG
    assert ws_status([dict(layer(fk, 64, 128), reserved0=1)])[0] == M.MKOR_INVALID_ARG
    # both paths keep a d_in x d_out fp32 intermediate
    sizes = [ws_status([dict(layer(fk, 1024, 4096, dt=1), gemm_path=p)])[1] for p in (M.GEMM_FP32, M.GEMM_SPLIT)]
    assert min(sizes) >= 4 * 1024 * 4096 and abs(sizes[0] - sizes[1]) < (1 << 20)


def test_rank_r_layers(lib):
    fk = Fake()
    assert ws_status([layer(fk, 37, 100, rank=4)])[0] == M.MKOR_OK
    assert ws_status([layer(fk, 64, 96, rank=2, rows=16)])[0] == M.MKOR_UNSUPPORTED   # means are rank-1
    assert ws_status([layer(fk, 64, 128, rank=2, fdt=1)])[0] == M.MKOR_UNSUPPORTED    # fp32 factors only
    # the r vectors of a factor extend over d * r floats
    a, b = layer(fk, 64, 64, rank=3), layer(fk, 64, 64, rank=3)
    b["a"] = a["a"] + 64 * 4 * 2          # read-only vectors may be shared
    assert ws_status([a, b])[0] == M.MKOR_OK
    a = layer(fk, 64, 64, rank=3)
    a["dW"] = a["a"] + 64 * 4 * 2         # a writable buffer over the third vector
    assert ws_status([a])[0] == M.MKOR_INVALID_ARG
    # Gram partials and r-wide vectors: the rank-4 plan needs more workspace
    r1 = ws_status([layer(fk, 1024, 1024)])[1]
    r4 = ws_status([layer(fk, 1024, 1024, rank=4)])[1]
    assert r4 > r1



@pytest.mark.parametrize("kw,ok", [
    (dict(), True), (dict(kind=M.OPT_SGD), True), (dict(kind=3), False), (dict(lr=-1.0), False),
    (dict(lr=math.inf), False), (dict(weight_decay=-0.1), False), (dict(kind=M.OPT_SGD, momentum=1.0), False),
    (dict(beta1=1.0), False), (dict(beta2=-0.1), False), (dict(eps=0.0), False), (dict(step=0), False),
    (dict(kind=M.OPT_SGD, step=0), True),
])
def test_opt_params(lib, kw, ok):
    st = M.opt_params_check(M.OptParams(**kw))
    assert (st == M.MKOR_OK) == ok, (kw, st, M.last_error())


def test_opt_buffers_validated(lib):
    fk = Fake()
    L = layer(fk, 64, 96)
    L.update(W=fk.alloc(64 * 96 * 4), opt_m=fk.alloc(64 * 96 * 4), opt_v=fk.alloc(64 * 96 * 4))
    assert ws_status([L])[0] == M.MKOR_OK
    L2 = dict(L)
    L2["opt_m"] = L["W"] + 64                 # state over the weights
    assert ws_status([L2])[0] == M.MKOR_INVALID_ARG
    L3 = dict(L)
    L3["W"] = L["G"]                          # weights over the (read-only) gradient
    assert ws_status([L3])[0] == M.MKOR_INVALID_ARG
    L4 = dict(L)
    L4["opt_v"] = L["opt_v"] + 4              # misaligned
    assert ws_status([L4])[0] == M.MKOR_INVALID_ARG


def test_noalloc_rejects_before_device(lib):
    """mkor_step_noalloc validates on the host and refuses a layer list larger
    than its device array before any HIP call."""
    fk = Fake()
    p = M.Params().to_c()
    assert lib.mkor_step_noalloc(None, 0, ctypes.byref(p), None) == M.MKOR_OK
    assert lib.mkor_step_noalloc(None, 0, None, None) == M.MKOR_INVALID_ARG
    big = B.make_layer_array([layer(fk, 4096, 4096)])   # its X alone is 64 MiB
    st, need = ws_status([layer(fk, 4096, 4096)])
    assert st == M.MKOR_OK and need > B.NOALLOC_MAX_BYTES
    assert lib.mkor_step_noalloc(big, 1, ctypes.byref(p), None) == M.MKOR_WORKSPACE_TOO_SMALL
    assert "mkor_step_noalloc" in M.last_error()
    bad = M.Params(gamma=2.0).to_c()
    small = [layer(fk, 64, 64)]
    assert lib.mkor_step_noalloc(B.make_layer_array(small), 1, ctypes.byref(bad), None) == M.MKOR_INVALID_ARG
    small[0]["dW"] = small[0]["G"]   # output aliases an input
    assert lib.mkor_step_noalloc(B.make_layer_array(small), 1, ctypes.byref(p), None) == M.MKOR_INVALID_ARG
    rk = [layer(fk, 64, 64, rank=2)]   # rank-r layers need the EXACT variant
    eq6 = M.Params(variant=M.SM_PAPER_EQ6).to_c()
    assert lib.mkor_step_noalloc(B.make_layer_array(rk), 1, ctypes.byref(eq6), None) == M.MKOR_UNSUPPORTED


def header_defines():
    """Integer #defines of include/mkor.h (name -> value)."""
    src = open(os.path.join(ROOT, "include", "mkor.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    out = {}
    for name, expr in re.findall(r"^#define\s+(MKOR_[A-Z0-9_]+)\s+(.+?)\s*$", src, flags=re.M):
        expr = expr.replace("u", "") if re.fullmatch(r"[0-9u<() ]+", expr) else expr
        try:
            out[name] = int(eval(expr, {"__builtins__": {}}))
        except Exception:
            pass
    return out


def test_binding_constants_match_header():
    d = header_defines()
    pairs = {
        "MKOR_ABI_VERSION": B.ABI_VERSION, "MKOR_OK": M.MKOR_OK, "MKOR_INVALID_ARG": M.MKOR_INVALID_ARG,
        "MKOR_WORKSPACE_TOO_SMALL": M.MKOR_WORKSPACE_TOO_SMALL, "MKOR_UNSUPPORTED": M.MKOR_UNSUPPORTED,
        "MKOR_HIP_ERROR": M.MKOR_HIP_ERROR, "MKOR_SM_EXACT": B.SM_EXACT, "MKOR_SM_PAPER_EQ6": B.SM_PAPER_EQ6,
        "MKOR_NORM_INF": B.NORM_INF, "MKOR_NORM_MAXABS": B.NORM_MAXABS, "MKOR_DTYPE_F32": B.DTYPE_F32,
        "MKOR_DTYPE_BF16": B.DTYPE_BF16, "MKOR_STAGE_MEANS": B.STAGE_MEANS, "MKOR_STAGE_SM_PASS": B.STAGE_SM_PASS,
        "MKOR_STAGE_SM_FINALIZE": B.STAGE_SM_FINALIZE, "MKOR_STAGE_GEMM_PREP": B.STAGE_GEMM_PREP,
        "MKOR_STAGE_GEMM_XT": B.STAGE_GEMM_XT, "MKOR_STAGE_GEMM_DW": B.STAGE_GEMM_DW,
        "MKOR_STAGE_RESCALE": B.STAGE_RESCALE, "MKOR_NUM_STAGES": B.NUM_STAGES, "MKOR_GEMM_AUTO": B.GEMM_AUTO,
        "MKOR_GEMM_FP32": B.GEMM_FP32, "MKOR_GEMM_SPLIT": B.GEMM_SPLIT, "MKOR_MAX_DIM": B.MAX_DIM,
        "MKOR_MAX_ROWS": B.MAX_ROWS, "MKOR_MAX_RANK": B.MAX_RANK, "MKOR_OPT_SGD": B.OPT_SGD,
        "MKOR_OPT_LAMB": B.OPT_LAMB, "MKOR_NOALLOC_MAX_BYTES": B.NOALLOC_MAX_BYTES,
    }
    assert set(d) == set(pairs), sorted(set(d) ^ set(pairs))
    for name, value in pairs.items():
        assert d[name] == value, (name, d[name], value)
    stages = sorted((v, k) for k, v in d.items() if k.startswith("MKOR_STAGE_"))
    assert [k[len("MKOR_STAGE_"):].lower() for _, k in stages] == B.STAGE_NAMES


def test_hybrid_struct_sizes():
    assert ctypes.sizeof(B.mkor_hybrid_params) == 16
    assert ctypes.sizeof(B.mkor_hybrid_state) == 16 + 3 * 8 + 2 * 8 + 4 * 4


def test_mode_and_pending_calls_on_host(lib):
    flags = (ctypes.c_int32 * 1)(1)
    out = ctypes.c_int32(5)
    assert lib.mkor_set_second_order(None, flags, None) == M.MKOR_INVALID_ARG
    assert lib.mkor_factors_pending(None, ctypes.byref(out)) == M.MKOR_INVALID_ARG
    plan = ctypes.c_void_p(None)
    assert lib.mkor_plan_create(None, 0, None, 0, ctypes.byref(plan)) == M.MKOR_OK
    assert lib.mkor_set_second_order(plan, None, None) == M.MKOR_OK   # n = 0: nothing to set
    assert lib.mkor_factors_pending(plan, None) == M.MKOR_INVALID_ARG
    assert lib.mkor_factors_pending(plan, ctypes.byref(out)) == M.MKOR_OK and out.value == 0
    lib.mkor_plan_destroy(plan)


def test_entry_points_open_roctx_ranges(lib):
    """The library imports roctx's range calls (each entry point opens a
    named range for traces taken with rocprofv3 --marker-trace)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", M.LIB_PATH], capture_output=True, text=True).stdout
    assert "roctxRangePushA" in out and "roctxRangePop" in out


# ------------------------------------------------------------------ property-based fuzz of validation

from hypothesis import HealthCheck, given, settings, strategies as hst  # noqa: E402

FUZZ_DIMS = [-1, 0, 1, 3, 37, 64, 100, 128, 192, 1024, M.MAX_DIM, M.MAX_DIM + 1]
PTR_KEYS = ["Linv", "Rinv", "a", "g", "G", "dW", "stats", "A", "Gout"]


def _mutate(L, other, kind, key):
    if kind == "null" and key in PTR_KEYS:
        L[key] = None
    elif kind == "misalign" and key in PTR_KEYS and L.get(key):
        L[key] += 4
    elif kind == "alias_out":
        L["dW"] = L["G"]
    elif kind == "overlap_factors":
        L["Rinv"] = L["Linv"] + 256
    elif kind == "cross_layer" and other is not None:
        L["dW"] = other["dW"]
    elif kind == "bad_code":
        L[key if key in ("grad_dtype", "factor_dtype", "act_dtype", "gemm_path", "second_order")
          else "grad_dtype"] = 7


def _valid_layer(fk, data):
    """A layer that satisfies every documented constraint."""
    d_in, d_out = (data.draw(hst.sampled_from([1, 3, 37, 64, 100, 128, 192, 1024])) for _ in range(2))
    m64 = d_in % 64 == 0 and d_out % 64 == 0
    so = data.draw(hst.sampled_from([0, 1, 1]))
    rows = data.draw(hst.sampled_from([0, 0, 1, 128]))
    fdt = data.draw(hst.sampled_from([0, 1])) if m64 else 0
    rank = data.draw(hst.sampled_from([0, 1, 2, 4])) if (so and fdt == 0 and rows == 0) else 0
    L = layer(fk, d_in, d_out, so=so, dt=data.draw(hst.sampled_from([0, 1])), stats=data.draw(hst.booleans()),
              rows=rows, adt=data.draw(hst.sampled_from([0, 1])), fdt=fdt, rank=rank)
    L["gemm_path"] = data.draw(hst.sampled_from([0, 1, 2] if m64 else [0, 1]))
    return L


def _random_layer(fk, data, prev):
    """A layer with random, often out-of-range values and up to two mutations."""
    d_in, d_out = data.draw(hst.sampled_from(FUZZ_DIMS)), data.draw(hst.sampled_from(FUZZ_DIMS))
    rows = data.draw(hst.sampled_from([0, 0, 0, 1, 128]))
    L = layer(fk, max(d_in, 1), max(d_out, 1), so=data.draw(hst.sampled_from([0, 1, 1, 1, 2])),
              dt=data.draw(hst.sampled_from([0, 1])), stats=data.draw(hst.booleans()), rows=rows,
              adt=data.draw(hst.sampled_from([0, 1])), fdt=data.draw(hst.sampled_from([0, 0, 1])),
              rank=data.draw(hst.sampled_from([0, 0, 1, 2, 4, 5, -1])))
    L["d_in"], L["d_out"] = d_in, d_out
    L["gemm_path"] = data.draw(hst.sampled_from([0, 0, 1, 2, 3, -1]))
    if data.draw(hst.booleans()):
        L["rows"] = data.draw(hst.sampled_from([-1, 8, M.MAX_ROWS + 1]))
    for _ in range(data.draw(hst.integers(1, 2))):
        _mutate(L, prev,
                data.draw(hst.sampled_from(["null", "misalign", "alias_out", "overlap_factors", "cross_layer",
                                            "bad_code"])),
                data.draw(hst.sampled_from(PTR_KEYS + ["gemm_path", "act_dtype", "factor_dtype"])))
    return L


@settings(max_examples=400, deadline=None, derandomize=True, suppress_health_check=list(HealthCheck))
@given(data=hst.data())
def test_validation_fuzz(lib, data):
    """Random layer lists (two thirds of the layers valid by construction, the
    others with out-of-range values, null or misaligned pointers, aliasing):
    mkor_workspace_size returns a documented status (and the error text on
    failure), the same size on a repeated call, a multiple of 256 B; plan
    creation with one byte too little workspace is refused with
    MKOR_WORKSPACE_TOO_SMALL before any HIP call."""
    fk = Fake()
    descs = []
    for _ in range(data.draw(hst.integers(0, 4), label="n")):
        ok = data.draw(hst.sampled_from([True, True, False]))
        descs.append(_valid_layer(fk, data) if ok else _random_layer(fk, data, descs[-1] if descs else None))
    st, size = ws_status(descs)
    assert st in (M.MKOR_OK, M.MKOR_INVALID_ARG, M.MKOR_UNSUPPORTED), (st, M.last_error())
    if st != M.MKOR_OK:
        assert M.last_error()
        return
    assert ws_status(descs) == (st, size)
    assert size % 256 == 0
    if size > 0:
        arr = B.make_layer_array(descs)
        plan = ctypes.c_void_p(None)
        ws = fk.alloc(size)
        assert lib.mkor_plan_create(arr, len(descs), ctypes.c_void_p(ws), size - 1,
                                    ctypes.byref(plan)) == M.MKOR_WORKSPACE_TOO_SMALL
        assert not plan.value


@settings(max_examples=300, deadline=None, derandomize=True, suppress_health_check=list(HealthCheck))
@given(gamma=hst.floats(allow_nan=True, allow_infinity=True, width=32),
       zeta=hst.floats(allow_nan=True, allow_infinity=True, width=32),
       eps=hst.floats(allow_nan=True, allow_infinity=True, width=32),
       norm_kind=hst.integers(-1, 2), variant=hst.integers(-1, 2))
def test_params_fuzz(lib, gamma, zeta, eps, norm_kind, variant):
    """mkor_params_check against the documented ranges: 0 < gamma < 1,
    0 < zeta <= 1, eps >= 0 (or +inf), norm kind and variant 0 or 1."""
    p = M.Params(gamma=gamma, zeta=zeta, eps=eps, norm_kind=norm_kind, variant=variant)
    valid = (0 < gamma < 1 and 0 < zeta <= 1 and (eps >= 0 or eps == math.inf) and not math.isnan(eps)
             and norm_kind in (0, 1) and variant in (0, 1))
    assert M.params_check(p) == (M.MKOR_OK if valid else M.MKOR_INVALID_ARG), (gamma, zeta, eps, M.last_error())
