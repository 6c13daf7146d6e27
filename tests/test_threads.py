"""The host side of the C interface from several threads at once (a plan
may be created, described and destroyed on any thread; the remembered
choices of gett_plan_tune sit in a shared table): concurrent planning gives
the same plans as serial planning.  CPU only; the sanitizer run covers it
too."""
import json
from concurrent.futures import ThreadPoolExecutor

import paper_1607_00145_amd as g
import workloads as wl
from workloads import appendix_a as ap


def shapes():
    ws = list(wl.WORKLOADS) + ap.appendix_workloads("f32")[:16] + ap.appendix_workloads("f64")[:16]
    return [(0 if w.dtype == "f32" else 1, w) for w in ws]


def describe(code, w):
    st, h = g.gett_plan(code, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, 0)
    assert st == 0, g.gett_status_string(st)
    try:
        d = json.loads(g.gett_plan_describe(h))
    finally:
        assert g.gett_destroy(h) == 0
    return json.dumps(d, sort_keys=True)


def test_concurrent_planning_matches_serial():
    cases = shapes()
    serial = [describe(c, w) for c, w in cases]
    jobs = [cases[i % len(cases)] for i in range(8 * len(cases))]
    with ThreadPoolExecutor(8) as ex:
        got = list(ex.map(lambda cw: describe(*cw), jobs))
    for i, d in enumerate(got):
        assert d == serial[i % len(cases)], cases[i % len(cases)][1].name


def test_concurrent_error_paths():
    """Refusals from many threads: statuses and texts stay right."""
    def bad(i):
        st, h = g.gett_plan(7 + i, "m,n", [2, 2], None, "m,k", [2, 2], None, "k,n", [2, 2], None)
        assert st == g.GETT_ERROR_INVALID_VALUE and h is None
        assert g.gett_status_string(st) == "invalid value"
        st, h = g.gett_plan(0, "m,n", [2, 3], None, "m,k", [2, 2], None, "k,n", [2, 2], None)
        assert st == g.GETT_ERROR_INVALID_INDICES and h is None
        return True
    with ThreadPoolExecutor(8) as ex:
        assert all(ex.map(bad, range(400)))
