"""The opt-in kernel timer (sp_profile_events), which the benchmark's
roofline figure rests on: the events bracket the armed kernel on the stream
of the call, describe its last launch, stay untouched once disarmed, and are
per calling thread."""
import threading

import numpy as np
import pytest

from tests.helpers import lib_desc, make_shard, to_dev
from workloads import shard_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _events(torch):
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    b.record()
    torch.cuda.synchronize()
    return a, b


def _problem(sp):
    sh = make_shard("timer", 2048, 2048, 128, 2, 0, 2, 2, 1, 2, 0, [2048], seed_base=9)
    q, k, v, do = (to_dev(x) for x in shard_inputs(sh))
    return lib_desc(sh), q, k, v, do


def test_events_bracket_the_kernel_on_the_call_stream(sp):
    import torch
    d, q, k, v, do = _problem(sp)
    sp.sp_attn_fwd(d, q, k, v)  # warm
    torch.cuda.synchronize()
    start, stop = _events(torch)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        mark = torch.cuda.Event(enable_timing=True)
        mark.record()
        torch.cuda._sleep(20_000_000)  # milliseconds of spinning before the call
        sp.sp_profile_events(sp.SP_KERNEL_ATTN_FWD, start, stop)
        try:
            sp.sp_attn_fwd(d, q, k, v)
        finally:
            sp.sp_profile_events(sp.SP_KERNEL_ATTN_FWD)
        after = torch.cuda.Event(enable_timing=True)
        after.record()
    s.synchronize()
    kernel_ms = start.elapsed_time(stop)
    # recorded on s after the spin, and before whatever follows on s
    assert mark.elapsed_time(start) > 1.0
    assert 0.0 < kernel_ms <= start.elapsed_time(after) + 1e-3
    # disarmed: a further launch leaves the events as they were
    sp.sp_attn_fwd(d, q, k, v)
    torch.cuda.synchronize()
    assert start.elapsed_time(stop) == kernel_ms


def test_events_describe_the_last_launch_and_are_per_thread(sp):
    import torch
    d, q, k, v, do = _problem(sp)
    o, lse = sp.sp_attn_fwd(d, q, k, v)
    torch.cuda.synchronize()
    start, stop = _events(torch)
    initial = start.elapsed_time(stop)
    sp.sp_profile_events(sp.SP_KERNEL_ATTN_DKDV, start, stop)
    try:
        # another thread's launches do not touch this thread's timer
        other = threading.Thread(target=lambda: (sp.sp_attn_bwd(d, q, k, v, o, lse, do),
                                                 torch.cuda.synchronize()))
        other.start()
        other.join(timeout=120)
        torch.cuda.synchronize()
        untouched = start.elapsed_time(stop)
        first = torch.cuda.Event(enable_timing=True)
        mid = torch.cuda.Event(enable_timing=True)
        first.record()
        sp.sp_attn_bwd(d, q, k, v, o, lse, do)
        mid.record()
        sp.sp_attn_bwd(d, q, k, v, o, lse, do)
        torch.cuda.synchronize()
    finally:
        sp.sp_profile_events(sp.SP_KERNEL_ATTN_DKDV)
    assert untouched == initial
    # the events describe the second call's dK/dV launch, which ends after
    # the marker recorded between the two calls
    assert first.elapsed_time(stop) > first.elapsed_time(mid)
    assert start.elapsed_time(stop) > 0.0
