"""The torch wrapper rejects tensors that do not match the plan before any
pointer reaches the C ABI (CPU tests: the ABI entry points are replaced by a
sentinel that fails if called, and the wrapper's device is the CPU)."""

import pytest
import torch

import paper_2605_30842_amd.binding as B

ABI = ("comem_decode_attn", "comem_decode_attn_paged", "comem_kv_append", "comem_kv_append_paged",
       "comem_append_decode_attn", "comem_append_decode_attn_paged", "comem_prefill_attn",
       "comem_prefill_attn_paged")


class Reached(Exception):
    pass


@pytest.fixture
def op(monkeypatch):
    def sentinel(*a, **k):
        raise Reached()

    for name in ABI:
        monkeypatch.setattr(B, name, sentinel)
    o = object.__new__(B.DecodeAttention)
    o.plan = None
    o.dtype = "bf16"
    o.num_q_heads, o.num_kv_heads, o.head_dim = 8, 2, 64
    o._torch_device = torch.device("cpu")
    o._q_dtypes, o._kv_dtypes = B._torch_dtypes("bf16")
    o.workspace = torch.zeros(256, dtype=torch.uint8)
    o.workspace_bytes = 256
    o._stream = staticmethod(lambda s: 0)
    return o


def _good(batch=3, T=40, paged=False):
    bf = torch.bfloat16
    d = dict(q=torch.zeros(batch, 8, 64, dtype=bf),
             ctx_lens=torch.tensor([5, 0, 7][:batch], dtype=torch.int32),
             out=torch.zeros(batch, 8, 64), lse=torch.zeros(batch, 8))
    if paged:
        d.update(k=torch.zeros(6, 16, 2, 64, dtype=bf), v=torch.zeros(6, 16, 2, 64, dtype=bf),
                 block_table=torch.zeros(batch, 4, dtype=torch.int32))
    else:
        d.update(k=torch.zeros(T, 2, 64, dtype=bf), v=torch.zeros(T, 2, 64, dtype=bf),
                 seq_start=torch.tensor([0, 10, 20][:batch], dtype=torch.int64))
    return d


def _forward(op, d):
    return op.forward(d["q"], d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64, out=d["out"], lse=d["lse"])


def _forward_paged(op, d):
    return op.forward_paged(d["q"], d["k"], d["v"], d["block_table"], d["ctx_lens"], 64, out=d["out"],
                            lse=d["lse"])


def test_valid_arguments_reach_the_abi(op):
    with pytest.raises(Reached):
        _forward(op, _good())
    with pytest.raises(Reached):
        _forward_paged(op, _good(paged=True))


BAD = {
    "q float32": ("q", lambda d: d["q"].float()),
    "q int64 lengths": ("ctx_lens", lambda d: d["ctx_lens"].long()),
    "ctx_lens short": ("ctx_lens", lambda d: d["ctx_lens"][:2]),
    "ctx_lens 2-D": ("ctx_lens", lambda d: d["ctx_lens"][None]),
    "seq_start int32": ("seq_start", lambda d: d["seq_start"].int()),
    "q wrong heads": ("q", lambda d: torch.zeros(3, 4, 64, dtype=torch.bfloat16)),
    "q wrong head_dim": ("q", lambda d: torch.zeros(3, 8, 128, dtype=torch.bfloat16)),
    "q not contiguous": ("q", lambda d: torch.zeros(8, 3, 64, dtype=torch.bfloat16).transpose(0, 1)),
    "out bf16": ("out", lambda d: d["out"].bfloat16()),
    "out wrong batch": ("out", lambda d: torch.zeros(2, 8, 64)),
    "out not contiguous": ("out", lambda d: torch.zeros(64, 8, 3).permute(2, 1, 0)),
    "lse float64": ("lse", lambda d: d["lse"].double()),
    "lse wrong shape": ("lse", lambda d: torch.zeros(3, 4)),
    "k float32": ("k", lambda d: d["k"].float()),
    "k wrong kv heads": ("k", lambda d: torch.zeros(40, 4, 64, dtype=torch.bfloat16)),
    "k strided last dim": ("k", lambda d: torch.zeros(40, 2, 128, dtype=torch.bfloat16)[:, :, ::2]),
    "v other strides": ("v", lambda d: torch.zeros(40, 4, 64, dtype=torch.bfloat16)[:, :2]),
    "q on meta": ("q", lambda d: d["q"].to("meta")),
    "ctx_lens a list": ("ctx_lens", lambda d: [5, 0, 7]),
}


@pytest.mark.parametrize("case", sorted(BAD))
def test_contiguous_call_rejects(op, case):
    d = _good()
    key, make = BAD[case]
    d[key] = make(d)
    with pytest.raises(ValueError):
        _forward(op, d)


BAD_PAGED = {
    "block_table int64": ("block_table", lambda d: d["block_table"].long()),
    "block_table rows": ("block_table", lambda d: d["block_table"][:2]),
    "block_table 1-D": ("block_table", lambda d: d["block_table"].flatten()),
    "k_pages 3-D": ("k", lambda d: d["k"][0]),
    "ctx_lens int64": ("ctx_lens", lambda d: d["ctx_lens"].long()),
}


@pytest.mark.parametrize("case", sorted(BAD_PAGED))
def test_paged_call_rejects(op, case):
    d = _good(paged=True)
    key, make = BAD_PAGED[case]
    d[key] = make(d)
    with pytest.raises(ValueError):
        _forward_paged(op, d)


def test_max_ctx_len_must_be_an_integer(op):
    d = _good()
    with pytest.raises(ValueError):
        op.forward(d["q"], d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64.0)


def test_append_rejects_new_rows(op):
    d = _good()
    nk = torch.zeros(3, 2, 64, dtype=torch.bfloat16)
    with pytest.raises(Reached):
        op.append(nk, nk.clone(), d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64)
    for bad in (nk.float(), torch.zeros(3, 2, 32, dtype=torch.bfloat16), torch.zeros(2, 2, 64, dtype=torch.bfloat16)):
        with pytest.raises(ValueError):
            op.append(bad, bad, d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64)
    with pytest.raises(ValueError):
        op.append_forward(d["q"], nk, nk[:, :1], d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64)


def test_prefill_checks(op):
    d = _good()
    q = torch.zeros(12, 8, 64, dtype=torch.bfloat16)
    qs = torch.tensor([0, 5, 5], dtype=torch.int64)
    ql = torch.tensor([5, 0, 7], dtype=torch.int32)
    with pytest.raises(Reached):
        op.prefill(q, qs, ql, 7, d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64)
    for args in ((q, qs.int(), ql), (q, qs, ql.long()), (q.float(), qs, ql), (q, qs[:2], ql)):
        with pytest.raises(ValueError):
            op.prefill(*args, 7, d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64)
    with pytest.raises(ValueError):
        op.prefill(q, qs, ql, 7, d["k"], d["v"], d["seq_start"], d["ctx_lens"], 64, out=torch.zeros(12, 8, 64,
                                                                                                   dtype=torch.float64))


def test_fp8_plan_takes_bf16_queries_and_byte_caches(op):
    op.dtype = "fp8"
    op._q_dtypes, op._kv_dtypes = B._torch_dtypes("fp8")
    d = _good()
    d["k"] = torch.zeros(40, 2, 64, dtype=torch.uint8)
    d["v"] = torch.zeros(40, 2, 64, dtype=torch.uint8)
    with pytest.raises(Reached):
        _forward(op, d)
    d["q"] = d["q"].to(torch.uint8)
    with pytest.raises(ValueError):
        _forward(op, d)
