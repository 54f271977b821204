"""Seeded synthetic inputs for the batched multi-adapter LoRA delta.

This module only draws random numbers and rounds them to the storage dtype.
None of the delta's arithmetic lives here, so the HIP path and the CPU oracle
can both take their inputs from it without sharing any computation.

Shapes follow the paper's setting: LoRA on the projections of Llama-2 layers
(Table "Model and GPU configurations": hidden 4096 / 5120 / 8192), adapter
factors A in R^{H1 x r} and B in R^{r x H2} (Section 2.1, Eq. 1), a skewed
adapter popularity (the MAF trace of Section 7.1, stood in for here by a
truncated Zipf law) and prompt segments mixed with single decode tokens in one
continuously batched step (Section 2.2).

Every array of 16-bit floats is held as raw ``uint16`` bit patterns so that
both sides read exactly the same bits.

Draw order, for one ``numpy.random.default_rng(seed)``:
  1. adapter ranks,
  2. adapter index per segment, then segment lengths,
  3. every distinct input tensor ``x``,
  4. for each projection, for each adapter: ``A`` then ``B``,
  5. for each projection: the base output ``y``,
  6. only for workloads of the fused base projection: for each projection,
     the base weight ``W`` [h_in, h_out] (the paper's H1 x H2 weight).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

F16 = 0
BF16 = 1
DTYPE_NAMES = {F16: "f16", BF16: "bf16"}


# ---------------------------------------------------------------------------
# storage-dtype rounding of generated inputs
# ---------------------------------------------------------------------------

def f32_to_f16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to IEEE binary16 (nearest-even); return the bits."""
    return np.ascontiguousarray(a, dtype=np.float32).astype(np.float16).view(np.uint16)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even); return the bits.

    Inputs are finite normal draws, so no NaN handling is needed.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    return ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)


def to_bits(a: np.ndarray, dtype: int) -> np.ndarray:
    return f32_to_f16_bits(a) if dtype == F16 else f32_to_bf16_bits(a)


def bits_to_f32(bits: np.ndarray, dtype: int) -> np.ndarray:
    """Exact widening of 16-bit patterns to float32 (for building test inputs)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    if dtype == F16:
        return bits.view(np.float16).astype(np.float32)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bits(rng: np.random.Generator, shape, std: float, dtype: int) -> np.ndarray:
    """N(0, std^2) drawn in float32, scaled, then rounded to the storage dtype."""
    z = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        z *= np.float32(std)
    return to_bits(z, dtype)


def zipf_probs(n: int, s: float = 1.1) -> np.ndarray:
    """Truncated Zipf over ids 0..n-1 with p_k proportional to (k+1)^-s."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


# ---------------------------------------------------------------------------
# workload containers
# ---------------------------------------------------------------------------

@dataclass
class Projection:
    name: str
    h_in: int
    h_out: int
    x: str                      # key of the input tensor in Workload.xs
    A: List[np.ndarray]         # per adapter, uint16 [h_in, r_g], row-major
    B: List[np.ndarray]         # per adapter, uint16 [r_g, h_out], row-major
    y: np.ndarray               # uint16 [n_rows, h_out], the base output x.W
    W: Optional[np.ndarray] = None   # uint16 [h_in, h_out]: the base weight (fused base workloads only)


@dataclass
class Workload:
    name: str
    dtype: int
    n_rows: int
    seg_offset: np.ndarray      # int32 [S+1]
    seg_adapter: np.ndarray     # int32 [S], -1 = no adapter
    ranks: np.ndarray           # int32 [N]
    scales: np.ndarray          # float32 [N]
    xs: Dict[str, np.ndarray]   # uint16 [n_rows, h]
    projections: List[Projection]
    description: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def n_adapters(self) -> int:
        return int(self.ranks.shape[0])

    def row_adapter(self) -> np.ndarray:
        """Adapter index of every row (int32 [n_rows])."""
        out = np.full(self.n_rows, -1, dtype=np.int32)
        for s in range(self.seg_adapter.shape[0]):
            out[self.seg_offset[s]:self.seg_offset[s + 1]] = self.seg_adapter[s]
        return out

    def projection(self, name: str) -> Projection:
        for p in self.projections:
            if p.name == name:
                return p
        raise KeyError(name)


def build_workload(
    *,
    name: str,
    seed: int,
    dtype: int,
    n_adapters: int,
    rank_set: Optional[Sequence[int]] = None,
    fixed_ranks: Optional[Sequence[int]] = None,
    seg_adapter: Optional[Sequence[int]] = None,
    seg_lens: Optional[Sequence[int]] = None,
    n_segments: Optional[int] = None,
    adapter_law: str = "given",
    zipf_s: float = 1.1,
    len_range: Optional[tuple] = None,
    projections: Sequence[tuple] = (("q_proj", 4096, 4096, "x"),),
    xs: Optional[Dict[str, int]] = None,
    scale: Optional[float] = None,
    description: str = "",
    base_weight: bool = False,
) -> Workload:
    """Draw one workload in the fixed draw order.

    ``projections`` lists (name, h_in, h_out, x_key); ``xs`` maps every x_key
    to its width (defaults to the h_in of the first projection that names it).
    ``scale=None`` means the per-adapter scale 16/r; otherwise a constant.
    ``adapter_law``: "given" (seg_adapter passed), "zipf", "uniform" or
    "identity" (segment s uses adapter s).
    """
    rng = np.random.default_rng(seed)

    # 1. ranks
    if fixed_ranks is not None:
        ranks = np.asarray(fixed_ranks, dtype=np.int32)
        assert ranks.shape[0] == n_adapters
    else:
        ranks = rng.choice(np.asarray(rank_set, dtype=np.int32), size=n_adapters).astype(np.int32)

    # 2. adapter index per segment, then segment lengths
    if adapter_law == "given":
        sa = np.asarray(seg_adapter, dtype=np.int32)
    else:
        assert n_segments is not None
        if adapter_law == "zipf":
            sa = rng.choice(n_adapters, size=n_segments, p=zipf_probs(n_adapters, zipf_s)).astype(np.int32)
        elif adapter_law == "uniform":
            sa = rng.integers(0, n_adapters, size=n_segments).astype(np.int32)
        elif adapter_law == "identity":
            sa = np.arange(n_segments, dtype=np.int32)
        else:
            raise ValueError(adapter_law)
    if seg_lens is not None:
        lens = np.asarray(seg_lens, dtype=np.int64)
    elif len_range is not None:
        lens = rng.integers(len_range[0], len_range[1] + 1, size=sa.shape[0]).astype(np.int64)
    else:
        lens = np.ones(sa.shape[0], dtype=np.int64)
    assert lens.shape[0] == sa.shape[0]
    seg_offset = np.zeros(sa.shape[0] + 1, dtype=np.int32)
    seg_offset[1:] = np.cumsum(lens)
    n_rows = int(seg_offset[-1])

    if scale is None:
        scales = (16.0 / ranks.astype(np.float32)).astype(np.float32)
    else:
        scales = np.full(n_adapters, scale, dtype=np.float32)

    # 3. distinct inputs
    if xs is None:
        xs = {}
        for (_, h_in, _, xk) in projections:
            xs.setdefault(xk, h_in)
    x_arrays = {}
    for xk, width in xs.items():
        x_arrays[xk] = normal_bits(rng, (n_rows, width), 1.0, dtype)

    # 4. adapters, per projection then per adapter: A then B
    projs = []
    for (pname, h_in, h_out, xk) in projections:
        assert xs[xk] == h_in, (pname, xk)
        A_list, B_list = [], []
        for g in range(n_adapters):
            r = int(ranks[g])
            A_list.append(normal_bits(rng, (h_in, r), 1.0 / np.sqrt(h_in), dtype))
            B_list.append(normal_bits(rng, (r, h_out), 1.0 / np.sqrt(r), dtype))
        projs.append(Projection(pname, h_in, h_out, xk, A_list, B_list, None))

    # 5. base outputs
    for p in projs:
        p.y = normal_bits(rng, (n_rows, p.h_out), 1.0, dtype)

    # 6. base weights, W ~ N(0, 1/h_in) so that x.W ~ N(0, 1)
    if base_weight:
        for p in projs:
            p.W = normal_bits(rng, (p.h_in, p.h_out), 1.0 / np.sqrt(p.h_in), dtype)

    return Workload(
        name=name, dtype=dtype, n_rows=n_rows, seg_offset=seg_offset, seg_adapter=sa,
        ranks=ranks, scales=scales, xs=x_arrays, projections=projs, description=description,
    )


# ---------------------------------------------------------------------------
# the five named workloads (Llama-2 shapes)
# ---------------------------------------------------------------------------

def decode_q_proj_rank8(seed: int = 0) -> Workload:
    """Decode, one 4096->4096 q_proj, 8 tokens, 4 rank-8 adapters, token t uses
    adapter t % 4, fp16, constant scale 2.0."""
    return build_workload(
        name="decode_q4096_t8_r8x4_f16", seed=seed, dtype=F16, n_adapters=4,
        fixed_ranks=[8, 8, 8, 8], seg_adapter=[t % 4 for t in range(8)],
        projections=(("q_proj", 4096, 4096, "x"),), scale=2.0,
        description="decode q_proj 4096->4096, T=8, 4 adapters r=8, idx=t%4, fp16, s=2",
    )


def decode_mixed_rank(seed: int = 1) -> Workload:
    """Decode batch of 64 tokens on a 4096->4096 projection, 32 adapters with
    ranks uniform over {8,16,32,64}, adapter per token Zipf(1.1), fp16, 16/r."""
    return build_workload(
        name="decode_q4096_t64_mixed_rank_f16", seed=seed, dtype=F16, n_adapters=32,
        rank_set=[8, 16, 32, 64], adapter_law="zipf", n_segments=64,
        projections=(("q_proj", 4096, 4096, "x"),),
        description="decode q_proj 4096->4096, T=64, 32 adapters r in {8,16,32,64}, Zipf(1.1), fp16",
    )


def prefill_segments(seed: int = 2) -> Workload:
    """16 prompt segments, lengths uniform on [64,1024], one adapter per
    segment with rank in {8,16,32,64}, 4096->4096, bf16, 16/r."""
    return build_workload(
        name="prefill_q4096_16seg_bf16", seed=seed, dtype=BF16, n_adapters=16,
        rank_set=[8, 16, 32, 64], adapter_law="identity", n_segments=16,
        len_range=(64, 1024), projections=(("q_proj", 4096, 4096, "x"),),
        description="prefill 16 segments len U[64,1024], one adapter each, r in {8..64}, bf16",
    )


LLAMA13B_LAYER = (
    ("q_proj", 5120, 5120, "x_attn"),
    ("k_proj", 5120, 5120, "x_attn"),
    ("v_proj", 5120, 5120, "x_attn"),
    ("o_proj", 5120, 5120, "x_o"),
    ("gate_proj", 5120, 13824, "x_mlp"),
    ("up_proj", 5120, 13824, "x_mlp"),
    ("down_proj", 13824, 5120, "x_down"),
)


def llama13b_layer_decode(seed: int = 3) -> Workload:
    """One Llama-2-13B-shaped layer, 7 adapted projections, 128 decode tokens,
    64 adapters with ranks {8,16,32,64}, Zipf(1.1) adapter per token, bf16."""
    return build_workload(
        name="llama13b_layer_decode_t128_bf16", seed=seed, dtype=BF16, n_adapters=64,
        rank_set=[8, 16, 32, 64], adapter_law="zipf", n_segments=128,
        projections=LLAMA13B_LAYER,
        xs={"x_attn": 5120, "x_o": 5120, "x_mlp": 5120, "x_down": 13824},
        description="13B layer q,k,v,o 5120^2, gate,up 5120->13824, down 13824->5120; T=128 decode; 64 adapters",
    )


def llama70b_mixed_batch(seed: int = 4) -> Workload:
    """Continuous batch on Llama-2-70B shapes: q_proj 8192->8192 and gate
    8192->28672; 256 decode tokens then 4 prompt segments of 512 tokens; 128
    adapters with ranks {8,16,32,64,128}, Zipf(1.1), bf16. Both projections
    read the same input rows."""
    return build_workload(
        name="llama70b_mixed_256dec_4x512pre_bf16", seed=seed, dtype=BF16, n_adapters=128,
        rank_set=[8, 16, 32, 64, 128], adapter_law="zipf", n_segments=260,
        seg_lens=[1] * 256 + [512] * 4,
        projections=(("q_proj", 8192, 8192, "x"), ("gate_proj", 8192, 28672, "x")),
        description="70B q 8192^2 + gate 8192->28672; 256 decode + 4x512 prefill; 128 adapters r in {8..128}",
    )


def llama70b_mixed_batch_tp4(seed: int = 4) -> Workload:
    """One GPU's share of the 70B mixed batch under 4-way tensor parallelism
    (column-parallel q and gate: A replicated, B split by output columns):
    q_proj 8192->2048 and gate 8192->7168, the same batch, adapters and laws
    as llama70b_mixed_batch."""
    return build_workload(
        name="llama70b_mixed_tp4_shard_bf16", seed=seed, dtype=BF16, n_adapters=128,
        rank_set=[8, 16, 32, 64, 128], adapter_law="zipf", n_segments=260,
        seg_lens=[1] * 256 + [512] * 4,
        projections=(("q_proj", 8192, 2048, "x"), ("gate_proj", 8192, 7168, "x")),
        description="70B TP=4 shard: q 8192->2048 + gate 8192->7168; 256 decode + 4x512 prefill; 128 adapters",
    )


def prefill_base(seed: int = 2) -> Workload:
    """The prompt workload (16 segments, len U[64,1024], one adapter each, r in
    {8..64}, 4096->4096, bf16) with the base weight W of the projection: the
    whole of Eq. 1, y' = xW + s(xA)B, for the fused base projection."""
    return build_workload(
        name="prefill_base_q4096_16seg_bf16", seed=seed, dtype=BF16, n_adapters=16,
        rank_set=[8, 16, 32, 64], adapter_law="identity", n_segments=16,
        len_range=(64, 1024), projections=(("q_proj", 4096, 4096, "x"),), base_weight=True,
        description="prefill 16 segments + base weight: y = xW + s(xA)B, 4096->4096, bf16",
    )


def prefill_base_one_segment(seed: int = 5) -> Workload:
    """One prompt of 1024 tokens with one rank-64 adapter, 4096->4096, bf16,
    with the base weight: the single-prompt shape of the fused base projection."""
    return build_workload(
        name="prefill_base_l1024_r64_bf16", seed=seed, dtype=BF16, n_adapters=1,
        fixed_ranks=[64], seg_adapter=[0], seg_lens=[1024],
        projections=(("q_proj", 4096, 4096, "x"),), base_weight=True,
        description="one 1024-token prompt, rank 64, + base weight, 4096->4096, bf16",
    )


BASE_NAMED = {
    "prefill_base": prefill_base,
    "prefill_base_l1024": prefill_base_one_segment,
}


NAMED = {
    "decode_r8": decode_q_proj_rank8,
    "decode_mixed": decode_mixed_rank,
    "prefill": prefill_segments,
    "llama13b_layer": llama13b_layer_decode,
    "llama70b_mixed": llama70b_mixed_batch,
    "llama70b_mixed_tp4": llama70b_mixed_batch_tp4,
}


def small_random(
    seed: int,
    *,
    dtype: int,
    h_in: int,
    h_out: int,
    n_adapters: int,
    rank_set: Sequence[int],
    seg_lens: Sequence[int],
    seg_adapter: Sequence[int],
    scale: Optional[float] = None,
) -> Workload:
    """A one-projection workload of arbitrary shape for parity tests."""
    return build_workload(
        name=f"random_s{seed}", seed=seed, dtype=dtype, n_adapters=n_adapters,
        rank_set=rank_set, seg_adapter=seg_adapter, seg_lens=seg_lens,
        projections=(("proj", h_in, h_out, "x"),), scale=scale,
    )


# ---------------------------------------------------------------------------
# algorithmic traffic of one step (padding-free, distinct-adapter form)
# ---------------------------------------------------------------------------

def algorithmic_bytes(w: Workload, proj_names: Optional[Sequence[str]] = None, rows=None) -> int:
    """Bytes one pass must move at minimum: every distinct adapter referenced
    once (r*(h_in+h_out) elements per projection), every distinct x once, and
    y read and written once, over rows that carry an adapter.

    ``rows`` optionally restricts to a boolean row mask.
    """
    e = 2
    ra = w.row_adapter()
    active = ra >= 0
    if rows is not None:
        active = active & rows
    used = np.unique(ra[active])
    projs = [p for p in w.projections if proj_names is None or p.name in proj_names]
    n_act = int(active.sum())
    total = 0
    seen_x = set()
    for p in projs:
        total += sum(int(w.ranks[g]) * (p.h_in + p.h_out) for g in used) * e
        if p.x not in seen_x:
            seen_x.add(p.x)
            total += n_act * p.h_in * e
        total += n_act * 2 * p.h_out * e
    return total


def algorithmic_flops(w: Workload, proj_names: Optional[Sequence[str]] = None, rows=None) -> int:
    """2*r*(h_in+h_out) multiply-adds per adapted row per projection."""
    ra = w.row_adapter()
    active = ra >= 0
    if rows is not None:
        active = active & rows
    projs = [p for p in w.projections if proj_names is None or p.name in proj_names]
    r_rows = w.ranks[ra[active]].astype(np.int64)
    return int(sum(int((2 * r_rows * (p.h_in + p.h_out)).sum()) for p in projs))


def adapter_bytes_per_rank(shapes: Sequence[tuple], n_layers: int, elem_bytes: int = 2) -> int:
    """Bytes of one unit of rank for adapters on the given (h_in, h_out)
    projections of every layer."""
    return n_layers * sum((a + b) for a, b in shapes) * elem_bytes


# ---------------------------------------------------------------------------
# request traces for the scheduling simulation
# ---------------------------------------------------------------------------

def sim_trace(seed: int, n: int, rps: float, *, n_adapters: int = 64, rank_pool: Sequence[int] = (8, 16, 32, 64),
              zipf_s: float = 1.1, prompt: tuple = (16, 512), output: tuple = (16, 256)) -> List[dict]:
    """A seeded synthetic request trace (stand-in for a production trace):
    Poisson arrivals at ``rps`` requests per second, adapters drawn with Zipf
    popularity from a pool whose ranks are drawn uniformly from ``rank_pool``,
    prompt and output lengths uniform over the given inclusive ranges, and one
    uniform [0, 1) draw per request for a random router.

    Draw order, one ``numpy.random.default_rng(seed)``: adapter ranks,
    inter-arrival gaps, adapters, prompt lengths, output lengths, uniforms.
    Times are in milliseconds."""
    rng = np.random.default_rng(seed)
    ranks = rng.choice(np.asarray(rank_pool, dtype=np.int32), size=n_adapters)
    gaps = rng.exponential(1000.0 / rps, size=n)
    adapters = rng.choice(n_adapters, size=n, p=zipf_probs(n_adapters, zipf_s))
    prompts = rng.integers(prompt[0], prompt[1] + 1, size=n)
    outputs = rng.integers(output[0], output[1] + 1, size=n)
    us = rng.random(size=n)
    t = np.cumsum(gaps)
    return [dict(arrival=float(t[i]), rank=int(ranks[adapters[i]]), prompt=int(prompts[i]),
                 output=int(outputs[i]), u=float(us[i]), adapter=int(adapters[i])) for i in range(n)]
