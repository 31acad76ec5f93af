"""The five named workloads at full size, in the launch configuration the bench
times (automatic split plan, matrix-core kernel for bf16).

Every output and every lse of each workload is compared with the oracle's
whole-batch result (the multi-GB workloads included: the oracle streams one
(sequence, KV head) slice at a time and finishes them in seconds).
"""

import numpy as np
import pytest

import oracle.decode_attention as da
from tests.gpu_util import DeviceWorkload, check, make_op, run, say
from workloads.synth import WORKLOADS, generate

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_full_workload_every_output(i):
    import torch

    w = generate(WORKLOADS[i])
    say(f"case full workload {i} {w.spec.name} kv_bytes={w.kv_bytes}")
    dw = DeviceWorkload(w)
    out, lse = run(dw, make_op(w.spec))
    del dw
    torch.cuda.empty_cache()
    ro, rl = da.reference(w)
    err = check(out, lse, ro, rl, w.spec.dtype, w.spec.name)
    say(f"  max |err| {err:.3e}")


def test_headline_workload_repeated_calls_bitwise():
    """The batch-1 32K workload's 32 splits per KV head finish in an order
    that changes from call to call, so a different workgroup merges each
    head from call to call. Every call must give the same bits (the merge
    visits splits in index order), and the first must pass the gate."""
    w = generate(WORKLOADS[2])
    say(f"case repeated calls {w.spec.name}")
    dw = DeviceWorkload(w)
    op = make_op(w.spec)
    first = run(dw, op)
    ro, rl = da.reference(w)
    check(*first, ro, rl, w.spec.dtype, w.spec.name)
    for k in range(24):
        again = run(dw, op)
        assert np.array_equal(first[0], again[0]) and np.array_equal(first[1], again[1]), f"call {k + 1}"
