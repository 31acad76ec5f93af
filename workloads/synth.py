"""Seeded synthetic decode-attention workloads.

This module draws inputs and nothing else: random normals, the bf16 cast,
context lengths, page pools and block tables. It holds none of the attention
arithmetic, so both the CPU oracle's tests and the GPU path's tests and bench
can consume it without sharing any of the method's computation.

Shapes follow the paper's statement of the decode problem (Sec. 2.2, "LLM
Inference"): one new query token per sequence with ``h_q`` heads of size
``d_h``; a KV cache of ``l`` tokens per sequence with ``h_kv`` heads of size
``d_h``. For its decode profiling (Sec. 3.1) the paper feeds randomly drawn
inputs at a set context length and a batch size held fixed; the five named
workloads below stand in for that, with the shapes of the paper's models
(Qwen3-class GQA, head size 128).

Recipe (every choice that the paper leaves open):
  * seed of workload ``i`` is ``1000 + i``; ``SeedSequence(seed).spawn(6)``
    gives one independent stream each for [lengths, block table, q, k, v,
    key-scale mask], so adding a tensor never shifts the others;
  * q, K, V are N(0, 1) drawn as float32 (``standard_normal(dtype=float32)``)
    in flat chunks of 2**20 elements, chunk c from a generator seeded by the
    c-th child of that tensor's stream (so chunks can be drawn in parallel),
    and, for bf16 workloads, rounded to nearest-even to bfloat16;
  * "uniform in [a, b]" lengths are integers with both ends included;
  * the paged pool holds exactly ``sum_b ceil(L_b / page)`` pages (plus
    optional spares), handed out in the order of one random permutation;
    unused block-table entries are -1;
  * "5% of keys scaled x8" is a Bernoulli(0.05) draw per (pool token slot,
    KV head) row of K only; the whole head_dim vector is scaled before the
    bf16 cast (x8 is a power of two, so before/after the cast agree);
  * FP8 KV workloads (dtype "fp8"): q is drawn as for bf16; K and V are the
    same N(0, 1) draws divided by a per-tensor scale (k_scale, v_scale, a
    power of two by default, so the division is exact) and rounded to the
    nearest OCP FP8 E4M3 code (ties to even, by torch's float8_e4m3fn cast);
    the cache stores the codes and the scales travel with the workload.
"""

from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np

# Large tensors are drawn in chunks of this many elements, one child seed per
# chunk (part of the recipe: changing it changes the drawn values).
_DRAW_CHUNK = 1 << 20
_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))

STREAMS = ("lengths", "block_table", "q", "k", "v", "key_mask")


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    """Shape and distribution of one decode-attention workload."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str  # "f32" or "bf16" (q, K and V alike) or "fp8" (q bf16, K and V OCP FP8 E4M3 codes)
    lengths: tuple  # ("fixed", L) or ("uniform", lo, hi) or ("list", (L0, L1, ...))
    max_ctx_len: int  # upper bound on every length (planning / block-table width)
    layout: str = "contiguous"  # "contiguous" (packed ragged) or "paged"
    page_size: int = 0
    key_scale_frac: float = 0.0
    key_scale: float = 8.0
    seed: int = 0
    k_scale: float = 2.0 ** -6  # fp8 only: K = code value * k_scale
    v_scale: float = 2.0 ** -6  # fp8 only: V = code value * v_scale

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def scale(self) -> np.float32:
        """Softmax scale 1/sqrt(head_dim), as the float32 the kernels receive."""
        return np.float32(1.0 / math.sqrt(self.head_dim))

    @property
    def elem_bytes(self) -> int:
        """Bytes of one K or V element."""
        return {"f32": 4, "bf16": 2, "fp8": 1}[self.dtype]

    @property
    def q_dtype(self) -> str:
        return "bf16" if self.dtype == "fp8" else self.dtype

    def replace(self, **kw) -> "WorkloadSpec":
        return dataclasses.replace(self, **kw)


# The five named workloads (sizes as stated for this build's targets).
WORKLOADS = {
    1: WorkloadSpec("tiny_f32_L2048", 1, 8, 2, 64, "f32", ("fixed", 2048), 2048, seed=1001),
    2: WorkloadSpec("bf16_B1_L32768", 1, 32, 8, 128, "bf16", ("fixed", 32768), 32768, seed=1002),
    3: WorkloadSpec("bf16_ragged_B16_L4k-64k", 16, 32, 8, 128, "bf16",
                    ("uniform", 4096, 65536), 65536, seed=1003),
    4: WorkloadSpec("bf16_paged16_B64_L2k-16k", 64, 32, 8, 128, "bf16",
                    ("uniform", 2048, 16384), 16384, layout="paged", page_size=16,
                    key_scale_frac=0.05, seed=1004),
    5: WorkloadSpec("bf16_paged64_B8_L131072_G8", 8, 64, 8, 128, "bf16",
                    ("fixed", 131072), 131072, layout="paged", page_size=64, seed=1005),
    # FP8 KV variants of the headline and the longest shapes (KV quantization, an extension row)
    6: WorkloadSpec("fp8_B1_L32768", 1, 32, 8, 128, "fp8", ("fixed", 32768), 32768, seed=1006),
    7: WorkloadSpec("fp8_paged64_B8_L131072_G8", 8, 64, 8, 128, "fp8",
                    ("fixed", 131072), 131072, layout="paged", page_size=64, seed=1007),
}


def f32_to_fp8_e4m3_codes(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest OCP FP8 E4M3 code (ties to even) with torch's cast.

    Values must lie within the format's range (|x| <= 448); the codes are returned as uint8.
    """
    import torch

    x = np.ascontiguousarray(x, dtype=np.float32)
    if np.abs(x).max(initial=0.0) > 448.0:
        raise ValueError("value outside the FP8 E4M3 range")
    return torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    nan = np.isnan(x)
    # Non-NaN patterns are below 0xFF800001, so adding at most 0x8000 cannot wrap.
    r = ((np.where(nan, np.uint32(0), u) + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
         >> np.uint32(16)).astype(np.uint16)
    if nan.any():
        r[nan] = (u[nan] >> np.uint32(16)).astype(np.uint16) | np.uint16(0x0040)
    return r


def _draw_tensor(stream: np.random.SeedSequence, shape, dtype: str,
                 row_scale: Optional[np.ndarray] = None, quant_scale: float = 1.0) -> np.ndarray:
    """N(0,1) tensor drawn in fixed chunks of _DRAW_CHUNK elements.

    Chunk c is drawn from its own generator seeded by ``stream.spawn(n)[c]``, so
    the values depend only on the seed and the shape, never on the thread count.
    ``row_scale`` (optional) multiplies each row (all leading dims but the last)
    before the bf16 cast. For "fp8" the draws are divided by ``quant_scale``
    and rounded to FP8 E4M3 codes.
    """
    n = int(np.prod(shape))
    inner = shape[-1]
    assert _DRAW_CHUNK % inner == 0
    out = np.empty(n, dtype={"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[dtype])
    nchunks = max(1, -(-n // _DRAW_CHUNK))
    children = stream.spawn(nchunks)
    rs = None if row_scale is None else row_scale.reshape(-1)

    def work(c: int) -> None:
        lo = c * _DRAW_CHUNK
        hi = min(n, lo + _DRAW_CHUNK)
        x = np.random.default_rng(children[c]).standard_normal(hi - lo, dtype=np.float32)
        if rs is not None:
            x = (x.reshape(-1, inner) * rs[lo // inner: hi // inner, None]).reshape(-1)
        if dtype == "f32":
            out[lo:hi] = x
        elif dtype == "bf16":
            out[lo:hi] = f32_to_bf16_bits(x)
        else:
            out[lo:hi] = f32_to_fp8_e4m3_codes(x / np.float32(quant_scale))

    if nchunks == 1:
        work(0)
    else:
        with ThreadPoolExecutor(max_workers=min(_THREADS, nchunks)) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


@dataclasses.dataclass
class Workload:
    """Host arrays of one drawn workload (bf16 data held as uint16 bit patterns)."""

    spec: WorkloadSpec
    q: np.ndarray  # [B, Hq, D]
    ctx_lens: np.ndarray  # int32 [B]
    # contiguous layout
    k: Optional[np.ndarray] = None  # [T, Hkv, D]
    v: Optional[np.ndarray] = None
    seq_start: Optional[np.ndarray] = None  # int64 [B]
    # paged layout
    k_pages: Optional[np.ndarray] = None  # [P, page, Hkv, D]
    v_pages: Optional[np.ndarray] = None
    block_table: Optional[np.ndarray] = None  # int32 [B, max_pages], -1 padded

    @property
    def kv_bytes(self) -> int:
        """Algorithmic K+V bytes of one step: each K and V element of every context once."""
        s = self.spec
        return int(self.ctx_lens.astype(np.int64).sum()) * s.num_kv_heads * s.head_dim * 2 * s.elem_bytes


def draw_lengths(spec: WorkloadSpec, rng: np.random.Generator) -> np.ndarray:
    kind = spec.lengths[0]
    if kind == "fixed":
        lens = np.full(spec.batch, spec.lengths[1], dtype=np.int64)
    elif kind == "uniform":
        lens = rng.integers(spec.lengths[1], spec.lengths[2], size=spec.batch, endpoint=True)
    elif kind == "list":
        lens = np.asarray(spec.lengths[1], dtype=np.int64)
        assert lens.shape == (spec.batch,)
    else:
        raise ValueError(f"unknown length kind {kind!r}")
    assert lens.min(initial=0) >= 0 and lens.max(initial=0) <= spec.max_ctx_len
    return lens.astype(np.int32)


def generate(spec: WorkloadSpec, seed: Optional[int] = None, *, gap_rows: int = 0,
             spare_pages: int = 0, poison: bool = False) -> Workload:
    """Draw one workload.

    gap_rows:    contiguous layout only; rows left between consecutive sequences.
    spare_pages: paged layout only; pool pages that no sequence uses.
    poison:      fill every K/V row that no context covers (gaps, slots past
                 L_b in a last page, spare pages) with NaN, so that a kernel
                 that reads outside the contexts produces NaN.
    """
    seed = spec.seed if seed is None else seed
    seqs = dict(zip(STREAMS, np.random.SeedSequence(seed).spawn(len(STREAMS))))
    rng = {name: np.random.default_rng(s) for name, s in seqs.items()}
    B, Hq, Hkv, D = spec.batch, spec.num_q_heads, spec.num_kv_heads, spec.head_dim
    assert Hq % Hkv == 0
    lens = draw_lengths(spec, rng["lengths"])
    q = _draw_tensor(seqs["q"], (B, Hq, D), spec.q_dtype)
    nan_bits = {"f32": np.float32("nan"), "bf16": np.uint16(0x7FC0), "fp8": np.uint8(0x7F)}[spec.dtype]
    if spec.dtype == "fp8" and spec.key_scale_frac > 0:
        raise ValueError("scaled keys are not drawn for fp8 workloads")
    kq, vq = (spec.k_scale, spec.v_scale) if spec.dtype == "fp8" else (1.0, 1.0)

    if spec.layout == "contiguous":
        starts = np.zeros(B, dtype=np.int64)
        pos = 0
        for b in range(B):
            starts[b] = pos
            pos += int(lens[b]) + gap_rows
        T = max(pos, 1)
        rows = (T, Hkv)
        mask = None
        if spec.key_scale_frac > 0:
            mask = np.where(rng["key_mask"].random(rows) < spec.key_scale_frac,
                            np.float32(spec.key_scale), np.float32(1.0))
        k = _draw_tensor(seqs["k"], (T, Hkv, D), spec.dtype, mask, quant_scale=kq)
        v = _draw_tensor(seqs["v"], (T, Hkv, D), spec.dtype, quant_scale=vq)
        if poison:
            covered = np.zeros(T, dtype=bool)
            for b in range(B):
                covered[starts[b]: starts[b] + lens[b]] = True
            k[~covered] = nan_bits
            v[~covered] = nan_bits
        return Workload(spec, q, lens, k=k, v=v, seq_start=starts)

    if spec.layout != "paged":
        raise ValueError(spec.layout)
    ps = spec.page_size
    assert ps > 0
    pages_per_seq = [(int(L) + ps - 1) // ps for L in lens]
    used = sum(pages_per_seq)
    pool = used + spare_pages
    perm = rng["block_table"].permutation(pool).astype(np.int32)
    max_pages = (spec.max_ctx_len + ps - 1) // ps
    bt = np.full((B, max(max_pages, 1)), -1, dtype=np.int32)
    pos = 0
    for b in range(B):
        n = pages_per_seq[b]
        bt[b, :n] = perm[pos: pos + n]
        pos += n
    P = max(pool, 1)
    rows = (P, ps, Hkv)
    mask = None
    if spec.key_scale_frac > 0:
        mask = np.where(rng["key_mask"].random(rows) < spec.key_scale_frac,
                        np.float32(spec.key_scale), np.float32(1.0))
    kp = _draw_tensor(seqs["k"], (P, ps, Hkv, D), spec.dtype, mask, quant_scale=kq)
    vp = _draw_tensor(seqs["v"], (P, ps, Hkv, D), spec.dtype, quant_scale=vq)
    if poison:
        covered = np.zeros((P, ps), dtype=bool)
        for b in range(B):
            t = np.arange(int(lens[b]))
            covered[bt[b, t // ps], t % ps] = True
        kp[~covered] = nan_bits
        vp[~covered] = nan_bits
    return Workload(spec, q, lens, k_pages=kp, v_pages=vp, block_table=bt)


def draw_new_rows(spec: WorkloadSpec, seed: int):
    """The new token's key and value rows for every sequence: two [B, Hkv, D] tensors ~ N(0,1) in spec.dtype
    (fp8: divided by k_scale / v_scale and rounded to codes)."""
    ks, vs = np.random.SeedSequence(seed).spawn(2)
    shape = (spec.batch, spec.num_kv_heads, spec.head_dim)
    kq, vq = (spec.k_scale, spec.v_scale) if spec.dtype == "fp8" else (1.0, 1.0)
    return (_draw_tensor(ks, shape, spec.dtype, quant_scale=kq), _draw_tensor(vs, shape, spec.dtype, quant_scale=vq))


# ---------------------------------------------------------------- prefill workloads


@dataclasses.dataclass(frozen=True)
class PrefillSpec:
    """A cached-prefix prefill workload: the KV side is a WorkloadSpec whose
    lengths L_b count every cached token, the last M_b of them new.

    new_tokens: ("fixed", M), ("uniform", lo, hi), ("list", (M0, ...)) or
    ("all",) for M_b = L_b (an uncached prefill). M_b is capped at L_b.
    """

    name: str
    kv: WorkloadSpec
    new_tokens: tuple
    seed: int = 0


@dataclasses.dataclass
class PrefillWorkload:
    spec: PrefillSpec
    kv: Workload       # K/V, lengths, layout (its q is unused)
    q: np.ndarray      # [sum_b M_b, Hq, D], sequence b at q_start[b]
    q_start: np.ndarray  # int64 [B]
    q_lens: np.ndarray   # int32 [B]

    @property
    def score_count(self) -> int:
        """Visible (query token, key) pairs per query head: sum_b sum_i (L_b - M_b + i + 1)."""
        L = self.kv.ctx_lens.astype(np.int64)
        M = self.q_lens.astype(np.int64)
        return int(((L - M) * M + M * (M + 1) // 2).sum())

    @property
    def flops(self) -> int:
        """Algorithmic flops: 2 D for q.k and 2 D for p.v per visible pair and query head."""
        s = self.kv.spec
        return 4 * s.head_dim * s.num_q_heads * self.score_count


PREFILL_WORKLOADS = {
    1: PrefillSpec("bf16_prefill_B1_P32768_M1024",
                   WorkloadSpec("kv_B1_L33792", 1, 32, 8, 128, "bf16", ("fixed", 33792), 33792, seed=2001),
                   ("fixed", 1024), seed=2001),
    2: PrefillSpec("bf16_prefill_uncached_B1_L8192",
                   WorkloadSpec("kv_B1_L8192", 1, 32, 8, 128, "bf16", ("fixed", 8192), 8192, seed=2002),
                   ("all",), seed=2002),
    3: PrefillSpec("bf16_prefill_paged16_B8_L8k-32k_M128-2048",
                   WorkloadSpec("kv_B8_L8k-32k_paged16", 8, 32, 8, 128, "bf16", ("uniform", 8192, 32768), 32768,
                                layout="paged", page_size=16, seed=2003),
                   ("uniform", 128, 2048), seed=2003),
}


def generate_prefill(spec: PrefillSpec, seed: Optional[int] = None, **kv_kw) -> PrefillWorkload:
    """Draw the K/V side with ``generate`` (same recipe), then the new-token counts and queries.

    The counts and queries come from ``SeedSequence((seed, 1)).spawn(2)``, so
    the K/V side equals the decode draw of the same KV spec and seed.
    """
    seed = spec.seed if seed is None else seed
    kv = generate(spec.kv, seed=seed, **kv_kw)
    lens_ss, q_ss = np.random.SeedSequence((seed, 1)).spawn(2)
    rng = np.random.default_rng(lens_ss)
    B = spec.kv.batch
    kind = spec.new_tokens[0]
    if kind == "all":
        m = kv.ctx_lens.astype(np.int64)
    elif kind == "fixed":
        m = np.full(B, spec.new_tokens[1], dtype=np.int64)
    elif kind == "uniform":
        m = rng.integers(spec.new_tokens[1], spec.new_tokens[2], size=B, endpoint=True)
    elif kind == "list":
        m = np.asarray(spec.new_tokens[1], dtype=np.int64)
    else:
        raise ValueError(f"unknown new-token kind {kind!r}")
    m = np.minimum(m, kv.ctx_lens.astype(np.int64)).astype(np.int32)
    q_start = np.zeros(B, dtype=np.int64)
    q_start[1:] = np.cumsum(m.astype(np.int64))[:-1]
    total = int(m.astype(np.int64).sum())
    s = spec.kv
    q = _draw_tensor(q_ss, (max(total, 1), s.num_q_heads, s.head_dim), s.dtype)[:total]
    return PrefillWorkload(spec, kv, q, q_start, m)


def small_prefill_spec(base: PrefillSpec, ctx_lens: Sequence[int], new_tokens: Sequence[int], *,
                       seed: Optional[int] = None, **kw) -> PrefillSpec:
    """A prefill workload with the head shapes, dtype and layout of ``base`` but given lengths."""
    kv = small_spec(base.kv, ctx_lens, seed=seed, **kw)
    return PrefillSpec(base.name + "_small", kv, ("list", tuple(int(x) for x in new_tokens)),
                       seed=kv.seed if seed is None else seed)


def small_spec(base: WorkloadSpec, lengths: Sequence[int], *, max_ctx_len: Optional[int] = None,
               seed: Optional[int] = None, **kw) -> WorkloadSpec:
    """A workload with the head shapes, dtype and layout of ``base`` but given lengths."""
    lens = tuple(int(x) for x in lengths)
    mcl = max(lens) if max_ctx_len is None else max_ctx_len
    return base.replace(batch=len(lens), lengths=("list", lens), max_ctx_len=max(mcl, 1),
                        seed=base.seed if seed is None else seed, **kw)
