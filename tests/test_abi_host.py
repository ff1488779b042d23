"""Host-only checks of the C ABI library: it loads, exports every declared
symbol, validates its arguments, and builds tables identical to the oracle's
(no GPU needed)."""

import os
import re
import subprocess

import numpy as np
import pytest

from conftest import ROOT

dq = pytest.importorskip("paper_2609_19880_amd")
from oracle import tables as otab  # noqa: E402


def _declared():
    src = open(os.path.join(ROOT, "include", "dq.h")).read()
    return sorted(set(re.findall(r"\b(dq_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", dq.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (dq_[a-z_0-9]+)", out))
    declared = _declared()
    assert declared, "no declarations found"
    missing = [s for s in declared if s not in exported]
    assert not missing, missing


def test_no_alloc_scratch_size_matches_header():
    src = open(os.path.join(ROOT, "include", "dq.h")).read()
    m = re.search(r"#define DQ_NO_ALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", src)
    assert m, "DQ_NO_ALLOC_SCRATCH_BYTES not found"
    assert dq.DQ_NO_ALLOC_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))


def test_strerror():
    assert dq.dq_strerror(dq.DQ_OK) == "ok"
    assert "infeasible" in dq.dq_strerror(dq.DQ_ERR_INFEASIBLE)
    assert dq.dq_strerror(99) == "unknown error"


CONFIGS = [(128, 6, 12, 1.4, 36), (128, 5, 12, 1.4, 32), (128, 9, 12, 1.4, 48),
           (128, 17, 12, 1.4, 64), (128, 16, 12, 5.6, 36), (128, 16, 12, 8.6, 32),
           (128, 32, 12, 7.6, 48), (128, 64, 12, 7.8, 64), (128, 16, 12, 1.4, 36),
           (64, 4, 8, 1.4, 20), (256, 7, 10, 1.2, 80), (128, 2, 12, 1.0, 24),
           (128, 3, 9, 2.0, 30), (128, 64, 8, 1.4, 200), (1024, 6, 12, 1.4, 235),
           (1024, 8, 12, 1.4, 335), (512, 11, 11, 1.4, 150)]


@pytest.mark.parametrize("n,M,p,alpha,C", CONFIGS)
def test_tables_equal_oracle(n, M, p, alpha, C):
    info, t = dq.dq_compute_tables(n, M, p, C, alpha)
    ref = otab.build_tables(n, M, p, alpha, C)
    assert np.array_equal(t["freq"], ref.freq)
    assert np.array_equal(t["cum"], ref.cum)
    assert np.array_equal(t["cost"], ref.cost)
    assert np.array_equal(t["sym_of_z"], ref.sym_of_z)
    assert np.array_equal(t["lambda"], ref.lam)
    assert info.feasible == ref.feasible
    assert info.budget_q16 == ref.budget_q16
    assert info.min_cost_q16 == n * int(ref.cost.min())
    assert info.cheapest == ref.cheapest
    assert abs(info.expected_max - otab.expected_max_normal(n)) < 1e-11


def test_table2_boundary_through_the_library():
    """Tab. 2: 1024-value groups, 231 B value container (+4 B metadata)."""
    for M, ok in ((4, True), (6, True), (7, True), (8, True), (10, True), (11, True), (12, False), (14, False)):
        assert dq.dq_compute_tables(1024, M, 12, 235, 1.4)[0].feasible == ok
        assert dq.dq_compute_tables(1024, M, 12, 335, 1.4)[0].feasible
    for C, top in ((32, 7), (36, 9), (48, 14), (64, 28)):
        assert dq.dq_compute_tables(128, top, 12, C, 1.4)[0].feasible
        assert not dq.dq_compute_tables(128, top + 1, 12, C, 1.4)[0].feasible


@pytest.mark.parametrize("bad", [dict(head_dim=100), dict(head_dim=2048), dict(record_bytes=300), dict(levels=1), dict(levels=65),
                                 dict(precision_bits=7), dict(precision_bits=13), dict(record_bytes=8),
                                 dict(alpha=0.5), dict(alpha=float("nan"))])
def test_invalid_configs_rejected(bad):
    args = dict(head_dim=128, levels=6, precision_bits=12, record_bytes=36, alpha=1.4)
    args.update(bad)
    with pytest.raises(dq.DqError) as e:
        dq.dq_compute_tables(args["head_dim"], args["levels"], args["precision_bits"], args["record_bytes"],
                             args["alpha"])
    assert e.value.code == dq.DQ_ERR_INVALID_ARG


def test_smallest_feasible_alpha_matches_workloads():
    import dq_workloads as wl
    for (M, C), alpha in wl.LITERAL_ALPHA.items():
        assert dq.smallest_feasible_alpha(128, M, 12, C) == pytest.approx(alpha)


def test_workspace_size_grows_with_context():
    a = dq.dq_decode_workspace_bytes(16, 32, 8, 32768)
    b = dq.dq_decode_workspace_bytes(16, 32, 8, 65536)
    assert 0 < a <= b
    assert dq.dq_decode_workspace_bytes(0, 32, 8, 4096) == 0


def test_prerotated_flag_is_validated_and_leaves_tables_unchanged():
    import ctypes
    lib = dq._lib
    info = lib._Info()
    for flag, rc in ((0, dq.DQ_OK), (1, dq.DQ_OK), (2, dq.DQ_ERR_INVALID_ARG), (-1, dq.DQ_ERR_INVALID_ARG)):
        cfg = lib._Config(128, 6, 12, 36, 1.4, flag)
        assert lib._lib.dq_compute_tables(ctypes.byref(cfg), ctypes.byref(info), None, None, None, None,
                                          None) == rc
    a = dq.dq_compute_tables(128, 6, 12, 36, 1.4)[1]
    cfg = lib._Config(128, 6, 12, 36, 1.4, 1)
    freq = np.zeros(6, np.int32)
    assert lib._lib.dq_compute_tables(ctypes.byref(cfg), ctypes.byref(info), freq.ctypes.data, None, None, None,
                                      None) == dq.DQ_OK
    assert np.array_equal(freq, a["freq"])
