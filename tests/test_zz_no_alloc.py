"""The allocation-free decode call (library-held device scratch instead of a
caller workspace) through the C ABI: the same bits as comem_decode_attn with
the plan's workspace, and within the gate of the oracle, on consecutive calls
whose inputs shrink, across plans of different shapes and kernels."""

import numpy as np
import pytest

import oracle.decode_attention as da
import paper_2605_30842_amd.binding as B
from tests.gpu_util import DeviceWorkload, check, make_op, say
from workloads.synth import WORKLOADS, generate, small_spec

pytestmark = pytest.mark.gpu


def _pair(op, dw):
    """(workspace call, allocation-free call) outputs of one workload, as numpy arrays."""
    import torch

    s = dw.spec
    B_, Hq, D = dw.q.shape
    outs = []
    for noalloc in (False, True):
        out = torch.full((B_, Hq, D), float("nan"), dtype=torch.float32, device=dw.q.device)
        lse = torch.full((B_, Hq), float("nan"), dtype=torch.float32, device=dw.q.device)
        stream = torch.cuda.current_stream().cuda_stream
        args = (op.plan, dw.q.data_ptr(), dw.k.data_ptr(), dw.v.data_ptr(), dw.k.stride(0), dw.k.stride(1),
                dw.seq_start.data_ptr(), dw.ctx_lens.data_ptr(), B_, s.max_ctx_len, out.data_ptr(), lse.data_ptr())
        if noalloc:
            B.comem_decode_attn_noalloc(*args, stream)
        else:
            B.comem_decode_attn(*args, op.workspace.data_ptr(), op.workspace_bytes, stream)
        torch.cuda.synchronize()
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    return outs


def _case(op, spec, what):
    w = generate(spec)
    say(f"noalloc {what}: batch {spec.batch}, lengths {list(w.ctx_lens)[:6]}, dtype {spec.dtype}")
    (o_ws, l_ws), (o_na, l_na) = _pair(op, DeviceWorkload(w))
    assert np.array_equal(o_ws, o_na) and np.array_equal(l_ws, l_na), f"{what}: bits differ from the workspace call"
    ro, rl = da.reference(w)
    check(o_na, l_na, ro, rl, spec.dtype, what)


def test_noalloc_matches_workspace_call_on_shrinking_inputs():
    base = small_spec(WORKLOADS[3], [4096, 20000, 1, 33000, 0, 9000], seed=301, max_ctx_len=40000)
    op = make_op(base)
    _case(op, base, "first call")
    # a second, smaller call with the same plan: fewer sequences, shorter contexts
    _case(op, small_spec(WORKLOADS[3], [300, 2000], seed=302, max_ctx_len=40000), "second, smaller call")
    _case(op, small_spec(WORKLOADS[3], [1], seed=303, max_ctx_len=40000), "one token")


def test_noalloc_across_plans():
    """Plans of other shapes share the one scratch: their counters sit in the same fixed region, so a
    call never meets another plan's partial results where it expects zeros."""
    big = small_spec(WORKLOADS[3], [30000] * 12, seed=304, max_ctx_len=30000)
    _case(make_op(big), big, "12 x 30000 tokens")
    head = WORKLOADS[2]
    _case(make_op(head), head, "batch-1 32K workload")
    tiny = WORKLOADS[1]  # fp32, vector kernel
    _case(make_op(tiny), tiny, "fp32 2048 tokens")
    g8 = small_spec(WORKLOADS[5], [5000, 700], seed=305).replace(layout="contiguous", page_size=0)
    _case(make_op(g8), g8, "G=8 contiguous")
    # and back to a plan with few counters after one with many
    _case(make_op(head), small_spec(head, [17000], seed=306, max_ctx_len=32768), "batch-1 17000 tokens")


def test_noalloc_refuses_a_call_past_its_scratch():
    import torch

    spec = small_spec(WORKLOADS[3], [65536] * 64, seed=307)
    op = make_op(spec)
    dev = "cuda:0"
    q = torch.zeros((64, 32, 128), dtype=torch.bfloat16, device=dev)
    kv = torch.zeros((64, 8, 128), dtype=torch.bfloat16, device=dev)  # never read: the call is refused first
    ss = torch.zeros(64, dtype=torch.int64, device=dev)
    cl = torch.zeros(64, dtype=torch.int32, device=dev)
    out = torch.zeros((64, 32, 128), dtype=torch.float32, device=dev)
    st = B.load_library().comem_decode_attn_noalloc(op.plan, q.data_ptr(), kv.data_ptr(), kv.data_ptr(), 1024, 128,
                                                    ss.data_ptr(), cl.data_ptr(), 64, 65536, out.data_ptr(), None,
                                                    torch.cuda.current_stream().cuda_stream)
    assert st == B.ERR_SCRATCH_LIMIT
