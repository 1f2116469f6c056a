"""The stage timeline without a GPU: the default library has no stamps and
says so, the timeline build says it has them, and the tool's per-stage
summary reads a stamp array the way include/pctree_profile.h lays it out."""
from __future__ import annotations

import ctypes

import numpy as np

from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd import timeline as T


def test_default_library_has_no_timeline():
    assert P.lib().pctree_timeline_available() == 0
    buf = (ctypes.c_int64 * (P.TIMELINE_WHO * P.TIMELINE_STAGES * P.TIMELINE_EVENTS))()
    rate = ctypes.c_double()
    st = P.lib().pctree_timeline_read(ctypes.cast(buf, ctypes.c_void_p), ctypes.byref(rate))
    assert st == P.ERR_UNSUPPORTED


def test_timeline_build_reports_its_stamps():
    L = ctypes.CDLL(P.TIMELINE_LIB_PATH)
    L.pctree_timeline_available.restype = ctypes.c_int32
    assert L.pctree_timeline_available() == 1
    L.pctree_timeline_read.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]
    rate = ctypes.c_double()
    assert L.pctree_timeline_read(None, ctypes.byref(rate)) == P.ERR_INVALID_ARGUMENT


def _stamps():
    return np.full((P.TIMELINE_WHO, P.TIMELINE_STAGES, P.TIMELINE_EVENTS), np.nan)


def test_summary_of_a_single_launch_round():
    t = _stamps()
    for d in range(4):  # a stage every 10 us
        base = 10.0 * d
        t[T.FIRST, d, :4] = base + np.array([0.0, 1.0, 3.0, 4.0])
        t[T.LAST, d, :4] = base + np.array([0.2, 1.2, 3.1, 4.3])
        t[T.KEEPER, d, :3] = base + np.array([4.5, 6.0, 8.0])
    t[T.KEEPER, T.ROUND, :2] = [40.0, 49.0]
    r = T.summarize(t, 4)
    assert r["form"] == "single launch"
    assert r["stage_period_us"] == 10.0 and r["emission_us"] == 9.0 and r["round_us"] == 49.0
    s = r["stages"][2]
    assert (s["keeper_merge_us"], s["keeper_select_us"]) == (1.5, 2.0)
    assert (s["first_inputs_us"], s["first_stream_us"], s["first_publish_us"]) == (1.0, 2.0, 1.0)
    assert (s["last_inputs_us"], s["last_stream_us"], s["last_publish_us"]) == (1.0, 1.9, 1.2)
    assert s["selected_at_us"] == 28.0


def test_summary_of_per_stage_launches():
    t = _stamps()
    for d in (1, 2, 3):  # (stage 0 left unstamped: a stage of the narrow form)
        t[T.HEAD, d, :3] = 60.0 * d + np.array([0.0, 30.0, 35.0])
        t[T.MERGE, d, :3] = 60.0 * d + np.array([37.0, 44.0, 55.0])
    r = T.summarize(t, 4)
    assert r["form"] == "per-stage launches"
    assert [s["stage"] for s in r["stages"]] == [1, 2, 3]
    s = r["stages"][0]
    assert (s["head_stream_us"], s["head_us"], s["head_to_merge_us"]) == (30.0, 35.0, 2.0)
    assert (s["merge_rows_us"], s["merge_select_us"], s["stage_us"]) == (7.0, 11.0, 60.0)
    assert r["stages"][-1]["stage_us"] is None  # no next head launch
