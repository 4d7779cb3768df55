"""Plain CPU model of the kernel-to-bubble packing step (test infrastructure only).

Only the tests and the benchmark's reporting import this module; the product
library never does.

The bubble scheduler of the paper (§4.2, fine-grained bubble exploitation,
the ScheduleKernels step of the BubbleScheduler algorithm) places one
micro-batch's encoder computation, broken into kernels, into the LLM's
timeline: several kernels may share one bubble as long as their summed time
fits in the bubble, a kernel never starts before the one whose output it
reads (the chain's order is kept), and communication kernels are not put into bubbles but overlapped
with long LLM computation (§3.1, design decision 3; §4.2).

Reading used here (also stated in the design notes): the timeline is a list
of intervals in time order, each either a bubble (the GPU's compute stream is
idle) or a period of LLM computation; kernels are taken in chain order and
each goes, unsplit, into the earliest interval of its kind -- at or after the
interval of the kernel before it -- whose remaining time still holds it.
When a kernel finds no such interval, it and every later kernel stay
unplaced.
"""

__all__ = ["schedule_kernels", "feasible", "brute_force_assignments"]


def schedule_kernels(kernel_us, kernel_comm, interval_us, interval_bubble):
    """Return (interval index per kernel or -1, start offset in that interval or -1.0).

    kernel_us: durations in chain order; kernel_comm: True for a communication
    kernel; interval_us: interval lengths in time order; interval_bubble: True
    for a bubble, False for LLM computation.  Sums are formed in float64 in
    the order the kernels are placed.
    """
    n, m = len(kernel_us), len(interval_us)
    where = [-1] * n
    offset = [-1.0] * n
    cur = 0          # interval of the previous kernel (0 before the first)
    used = 0.0       # time already taken in interval `cur`
    for i in range(n):
        d = float(kernel_us[i])
        wants_bubble = not kernel_comm[i]
        placed = False
        for j in range(cur, m):
            if bool(interval_bubble[j]) != wants_bubble:
                continue
            start = used if j == cur else 0.0
            if start + d <= float(interval_us[j]):
                where[i], offset[i] = j, start
                cur, used = j, start + d
                placed = True
                break
        if not placed:
            break
    return where, offset


def feasible(assign, kernel_us, kernel_comm, interval_us, interval_bubble):
    """Whether a complete assignment keeps chain order, kinds and capacities."""
    if any(a < 0 for a in assign):
        return False
    if any(b < a for a, b in zip(assign, assign[1:])):
        return False
    load = {}
    for i, a in enumerate(assign):
        if bool(interval_bubble[a]) == bool(kernel_comm[i]):
            return False
        load[a] = load.get(a, 0.0) + float(kernel_us[i])
    return all(v <= float(interval_us[a]) for a, v in load.items())


def brute_force_assignments(kernel_us, kernel_comm, interval_us, interval_bubble):
    """Every feasible complete assignment (exhaustive; tiny inputs only)."""
    import itertools
    n, m = len(kernel_us), len(interval_us)
    out = []
    for assign in itertools.combinations_with_replacement(range(m), n):
        if feasible(list(assign), kernel_us, kernel_comm, interval_us, interval_bubble):
            out.append(list(assign))
    return out
