"""C-ABI checks that need no GPU: the library loads, exports every entry
point declared in include/esp.h, and rejects bad arguments on the host before
any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2608_07971_amd as esp
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "esp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(esp_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert {"esp_create", "esp_score_select", "esp_reduce_demand", "esp_update_prices", "esp_solve"} <= set(names)
    L = esp.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(esp._SIGS), "binding and header disagree"


def test_status_strings():
    for code in range(10):
        assert esp.status_string(code)
    assert esp.status_string(0) == "ok"


def _ws(p, opt=None):
    return esp.esp_workspace_size(p, opt)


def test_workspace_size_dense_and_csr():
    t = workloads.make("tiny")
    n1 = _ws(esp.Problem.from_instance(t))
    assert n1 >= t.table_bytes()
    r = workloads.make("ragged", n_jobs=5000)
    n2 = _ws(esp.Problem.from_instance(r))
    assert n2 >= r.table_bytes()
    L = workloads.make("large", n_jobs=1000)
    assert _ws(esp.Problem.from_instance(L)) >= L.table_bytes()


def test_workspace_size_profile_store():
    # the entry-major copy: each family's run rounded up to whole 128-byte
    # lines, B copies, plus a 64-byte directory record per 60 families (each
    # region aligned to 256 bytes)
    for inst in (workloads.make("tiny"), workloads.make("ragged", n_jobs=3000),
                 workloads.random_small(3, 301, 70, 8, n_clusters=3)):
        p = esp.Problem.from_instance(inst)
        base = _ws(p)
        more = _ws(p, esp.esp_options(0, 0, 0, esp.ESP_OPT_PROFILE_STORE))
        sizes = np.diff(np.asarray(inst.offsets, np.int64))
        lines = int(((sizes * 4 * (p.R + 1) + 127) // 128).sum())
        extra = p.B * lines * 128 + 64 * (-(-p.N // 60))
        assert extra <= more - base <= extra + 2 * 256


@pytest.mark.parametrize("field,value,code", [
    ("num_resources", 0, esp.ESP_ERR_SHAPE), ("num_resources", 9, esp.ESP_ERR_SHAPE),
    ("num_jobs", 0, esp.ESP_ERR_SHAPE), ("num_clusters", 0, esp.ESP_ERR_SHAPE),
    ("configs_per_job", 0, esp.ESP_ERR_SHAPE), ("configs_per_job", 257, esp.ESP_ERR_SHAPE),
])
def test_workspace_size_shape_errors(field, value, code):
    p = esp.Problem.from_instance(workloads.make("tiny"))
    setattr(p.c, field, value)
    with pytest.raises(esp.EspError) as e:
        _ws(p)
    assert e.value.code == code


def test_bad_offsets_and_options():
    inst = workloads.random_small(1, 10, 5, 2)
    p = esp.Problem.from_instance(inst)
    p.offsets[3] = p.offsets[2]                       # empty family
    with pytest.raises(esp.EspError) as e:
        _ws(p)
    assert e.value.code == esp.ESP_ERR_SHAPE
    p2 = esp.Problem.from_instance(inst)
    opt = esp.esp_options(0)
    opt.reserved[2] = 1
    opt2 = esp.esp_options(0, 5)
    with pytest.raises(esp.EspError) as e:
        _ws(p2, opt)
    assert e.value.code == esp.ESP_ERR_INVALID_ARG
    with pytest.raises(esp.EspError) as e:
        _ws(p2, esp.esp_options(0, 0, 0, 2))          # unknown flag
    assert e.value.code == esp.ESP_ERR_INVALID_ARG
    with pytest.raises(esp.EspError):
        _ws(p2, esp.esp_options(-1))
    with pytest.raises(esp.EspError):
        _ws(p2, opt2)


class _FakeWs:
    """Stands in for a workspace tensor in host-side rejection tests."""
    def __init__(self, ptr, n):
        self.ptr, self.n = ptr, n

    def numel(self):
        return self.n

    def element_size(self):
        return 1


def _create(inst, rule=None, eta0=None, ws_ptr=0, ws_n=0):
    p = esp.Problem.from_instance(inst)
    e0 = np.ascontiguousarray(inst.eta0 if eta0 is None else eta0, dtype=np.float64)
    step = esp.esp_step_rule(inst.rule if rule is None else rule, e0.ctypes.data)
    out = C.c_void_p(None)
    code = esp.lib().esp_create(C.addressof(p.c), C.addressof(step), None, ws_ptr or None, ws_n, None,
                                C.byref(out))
    return code, out.value


def test_create_rejects_bad_values_on_host():
    base = workloads.random_small(2, 8, 4, 3)
    nan_u = workloads.random_small(2, 8, 4, 3); nan_u.utility[0, 5] = np.nan
    inf_d = workloads.random_small(2, 8, 4, 3); inf_d.demand[0, 3, 1] = np.inf
    neg_d = workloads.random_small(2, 8, 4, 3); neg_d.demand[0, 3, 1] = -1.0
    nan_c = workloads.random_small(2, 8, 4, 3); nan_c.capacity[0, 0] = np.nan
    big_c = workloads.random_small(2, 8, 4, 3); big_c.capacity[0, 0] = 2.0 ** 300
    masked = workloads.random_small(2, 8, 4, 3)
    masked.feasible = np.ones((1, masked.nnz), np.uint8)
    masked.feasible[0, masked.offsets[2]:masked.offsets[3]] = 0
    wide = workloads.random_small(2, 8, 4, 3); wide.demand[0, 0, 0] = 1e-38; wide.demand[0, 1, 0] = 1e38
    assert _create(nan_u)[0] == esp.ESP_ERR_NONFINITE
    assert _create(inf_d)[0] == esp.ESP_ERR_NONFINITE
    assert _create(neg_d)[0] == esp.ESP_ERR_NEGATIVE_DEMAND
    assert _create(nan_c)[0] == esp.ESP_ERR_NONFINITE
    assert _create(big_c)[0] == esp.ESP_ERR_RANGE
    assert _create(masked)[0] == esp.ESP_ERR_EMPTY_FAMILY
    assert _create(wide)[0] == esp.ESP_ERR_RANGE
    assert _create(base, rule=7)[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(base, eta0=[0.0])[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(base, eta0=[np.inf])[0] == esp.ESP_ERR_NONFINITE
    assert _create(base, eta0=[2.0 ** 101])[0] == esp.ESP_ERR_RANGE
    # valid problem, missing / misaligned / short workspace
    assert _create(base)[0] == esp.ESP_ERR_WORKSPACE
    assert _create(base, ws_ptr=4096 + 8, ws_n=1 << 30)[0] == esp.ESP_ERR_WORKSPACE
    assert _create(base, ws_ptr=4096, ws_n=16)[0] == esp.ESP_ERR_WORKSPACE


def test_null_context_is_rejected():
    L = esp.lib()
    assert L.esp_solve(None, None, 1, 1, 0.0, None, None, None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_score_select(None, None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_reduce_demand(None, None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_update_prices(None, None, 1, None, None) == esp.ESP_ERR_STATE
    assert L.esp_device_status(None, None) == esp.ESP_ERR_STATE
    mode = C.c_int32(-1)
    assert L.esp_loop_driver(None, C.byref(mode)) == esp.ESP_ERR_STATE and mode.value == -1
    cap = (C.c_double * 2)(1.0, 2.0)
    assert L.esp_set_capacity(None, cap, None) == esp.ESP_ERR_STATE
    assert L.esp_effective_capacity(None, None, None, 0.5, None, None) == esp.ESP_ERR_STATE
    assert L.esp_nearest_profile(None, 1, None, None, None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_read_penalties(None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_schedule(None, None, 1, 1, 0.0, None, None, None, None, None, None) == esp.ESP_ERR_STATE
    assert L.esp_destroy(None) == esp.ESP_ERR_STATE


def test_create_rejects_bad_penalties_on_host():
    def mk():
        return workloads.with_penalties(workloads.random_small(9, 8, 4, 3), 9)
    neg = mk(); neg.penalty[0, 3] = -0.5
    nan = mk(); nan.penalty[0, 3] = np.nan
    cur = mk(); cur.current[0, 2] = 99
    sw = mk(); sw.switch_cost[:] = -1.0
    half = mk(); half.switch_cost = None
    assert _create(neg)[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(nan)[0] == esp.ESP_ERR_NONFINITE
    assert _create(cur)[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(sw)[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(half)[0] == esp.ESP_ERR_INVALID_ARG
    assert _create(mk())[0] == esp.ESP_ERR_WORKSPACE         # valid problem, no workspace
    assert esp.lib().esp_set_penalties(None, None, None, None, None) == esp.ESP_ERR_STATE


def test_workspace_grows_by_one_column_with_penalties():
    a = workloads.random_small(10, 50, 8, 3, dense=True)
    b = workloads.with_penalties(workloads.random_small(10, 50, 8, 3, dense=True), 10)
    na, nb = _ws(esp.Problem.from_instance(a)), _ws(esp.Problem.from_instance(b))
    assert nb - na >= 50 * 8 * 4


def test_resident_mode_refuses_tables_that_do_not_fit():
    """ESP_MODE_RESIDENT needs every wavefront to hold at most two tiles:
    refused with ESP_ERR_SHAPE before any device work (here: no workspace at
    all); a table that fits gets as far as the workspace check."""
    def create(inst, blocks):
        p = esp.Problem.from_instance(inst)
        e0 = np.ascontiguousarray(inst.eta0, dtype=np.float64)
        step = esp.esp_step_rule(inst.rule, e0.ctypes.data)
        opt = esp.esp_options(blocks, 0, esp.ESP_MODE_RESIDENT, 0)
        out = C.c_void_p(None)
        return esp.lib().esp_create(C.addressof(p.c), C.addressof(step), C.addressof(opt), None, 0, None,
                                    C.byref(out))
    small = workloads.make("small", n_jobs=200)          # 25 tiles
    assert create(small, 3) == esp.ESP_ERR_SHAPE          # 12 wavefronts hold at most 24
    assert create(small, 4) == esp.ESP_ERR_WORKSPACE
    assert create(workloads.make("tiny"), 0) == esp.ESP_ERR_WORKSPACE
    assert create(workloads.make("large", n_jobs=100000), 0) == esp.ESP_ERR_SHAPE
