"""The two tracebacks of rc_reconstruct, forced in turn through RCDP_TRACE.

"scan" walks optarg by scanning the predecessor list of each step's set
(k_trace); "slice" first derives optarg of every cell with t <= t* and then
follows it (k_trace_follow), within the slice's size limits: t* + 1 <= 65536,
fewer than 65535 sets and at most 2^24 cells.  Both must give the oracle's
schedule.
"""

import contextlib
import os

TRACES = ("scan", "slice")


@contextlib.contextmanager
def forced_trace(trace):
    old = os.environ.get("RCDP_TRACE")
    if trace is None:
        os.environ.pop("RCDP_TRACE", None)
    else:
        os.environ["RCDP_TRACE"] = trace
    try:
        yield
    finally:
        if old is None:
            os.environ.pop("RCDP_TRACE", None)
        else:
            os.environ["RCDP_TRACE"] = old


def expected_kernel(trace, num_sets, t_star):
    s = t_star + 1
    fits = s <= 65536 and num_sets < 65535 and num_sets * s <= 1 << 24
    return "k_trace_follow" if trace == "slice" and fits else "k_trace"


def reconstruct_each(sol, num_sets, traces=TRACES):
    """The schedule of every forced traceback, after checking which ran."""
    out = []
    for trace in traces:
        with forced_trace(trace):
            sched = sol.reconstruct()
        assert sol.trace_kernel() == expected_kernel(trace, num_sets, sol.t_star), trace
        out.append(sched)
    return out
