"""The progressive asynchronous schedule (Eq. 2, Alg. 2) through the C ABI:
step for step equal to the oracle's (phases, strides, intervals and the
double-precision alpha bit for bit), struct layout, counts and errors."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

rf = pytest.importorskip("paper_2606_06309_amd.binding")
lib = rf.lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_constants_and_layout_match_header():
    with open(os.path.join(ROOT, "include", "rhymeflow.h")) as f:
        text = f.read()
    for name in ("RF_STEP_WARMUP", "RF_STEP_RHYTHMIC", "RF_STEP_SKIP"):
        assert int(re.search(rf"#define {name} (\d+)", text).group(1)) == getattr(rf, name)
    body = re.search(r"typedef struct rf_step_plan \{(.*?)\} rf_step_plan;", text, re.S).group(1)
    fields = re.findall(r"^\s*(\w+)\s+(\w+);", body, re.M)
    assert [n for _, n in fields] == [n for n, _ in rf.rf_step_plan._fields_]
    assert ctypes.sizeof(rf.rf_step_plan) == 32


def test_matches_oracle():
    rng = np.random.default_rng(13)
    cases = [(50, 8, 25, 2, 3), (50, 8, 26, 2, 3), (10, 2, 4, 2, 3), (1, 0, 0, 1, 1), (1, 1, 1, 2, 3),
             (12, 12, 6, 2, 3), (6, 2, 0, 9, 9), (100, 15, 50, 2, 3), (40, 0, 40, 3, 2)]
    for _ in range(300):
        T = int(rng.integers(1, 120))
        cases.append((T, int(rng.integers(0, T + 1)), int(rng.integers(0, T + 1)),
                      int(rng.integers(1, 7)), int(rng.integers(1, 9))))
    for c in cases:
        got = rf.rf_async_schedule(*c)
        exp = oracle.async_schedule(*c)
        assert got == exp, c          # dict equality: alpha compared as doubles, exactly


def test_counts():
    plan = (rf.rf_step_plan * 50)()
    nr, ns = ctypes.c_int32(-1), ctypes.c_int32(-1)
    assert lib.rf_async_schedule(50, 8, 25, 2, 3, plan, ctypes.byref(nr), ctypes.byref(ns)) == rf.RF_OK
    assert (nr.value, ns.value) == (17, 25)
    assert lib.rf_async_schedule(50, 8, 25, 2, 3, plan, None, None) == rf.RF_OK


@pytest.mark.parametrize("args,status", [
    ((0, 0, 0, 2, 3), rf.RF_ERR_RANGE),
    ((1 << 21, 0, 0, 2, 3), rf.RF_ERR_RANGE),
    ((10, -1, 5, 2, 3), rf.RF_ERR_RANGE),
    ((10, 11, 5, 2, 3), rf.RF_ERR_RANGE),
    ((10, 2, 11, 2, 3), rf.RF_ERR_RANGE),
    ((10, 2, -1, 2, 3), rf.RF_ERR_RANGE),
    ((10, 2, 5, 0, 3), rf.RF_ERR_INVALID_ARG),
    ((10, 2, 5, 2, -3), rf.RF_ERR_INVALID_ARG),
])
def test_errors(args, status):
    plan = (rf.rf_step_plan * 16)()
    assert lib.rf_async_schedule(*args, plan, None, None) == status
    assert lib.rf_last_error().decode().startswith("rf_async_schedule")


def test_null_plan():
    assert lib.rf_async_schedule(10, 2, 5, 2, 3, None, None, None) == rf.RF_ERR_INVALID_ARG
