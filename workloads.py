"""Seeded synthetic inputs for the MoE block.

This module is shared by the oracle tests, the GPU parity tests and the bench.
It holds none of the block's arithmetic: only random draws, the bf16 encoding
of those draws, and the structural knobs of each workload (a router bias that
makes expert popularity Zipf-like, a padding mask from passage lengths).

Workloads (the reranker batches of the paper, §4.1 Setup: listwise groups of
query-passage pairs, bf16; and the Qwen3-30B-A3B expert layout of §3: 128
experts, top-8 routing):

* ``tiny``          T=256,  H=128,  E=8,   k=2, F=256   (seconds on the oracle)
* ``qwen3_30b_a3b`` T=8192, H=2048, E=128, k=8, F=768   (one GPU, near-uniform router)
* ``ep_share``      16 local experts, H=2048, F=768: the rows a T=8192, E=128,
                    k=8 routing sends to experts 0..15 (one expert-parallel
                    rank's share; 8359 rows, stored in tests/golden)
* ``zipf``          T=32768, qwen shape, router biased so that expert
                    popularity follows Zipf(s=1.2); 4 experts get no rows
* ``long_passage``  T=65536 = 16 passages x 4096 tokens, qwen shape, tokens
                    past each passage's length (~U{2048..4096}) masked out

All draws are fp32 from numpy's PCG64, split into fixed 4M-element chunks, each
chunk with its own child seed from ``SeedSequence(seed)``; results therefore do
not depend on how many threads generate them.  bf16 values are carried as
``uint16`` bit patterns (round-to-nearest-even from the fp32 draw).
"""
from __future__ import annotations

import json
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 22

CONFIGS = {
    "tiny": dict(kind="block", T=256, H=128, E=8, k=2, F=256, seed=0),
    "qwen3_30b_a3b": dict(kind="block", T=8192, H=2048, E=128, k=8, F=768, seed=1),
    "ep_share": dict(kind="experts", H=2048, E=16, F=768, seed=2,
                     E_total=128, k=8, T=8192),
    "zipf": dict(kind="block", T=32768, H=2048, E=128, k=8, F=768, seed=3,
                 zipf_s=1.2, zipf_scale=0.4, n_cold=4),
    "long_passage": dict(kind="block", T=65536, H=2048, E=128, k=8, F=768, seed=4,
                         passages=16, passage_len=4096, min_len=2048),
}

WEIGHT_STD = 0.02


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest even; NaN kept quiet."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> fp32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def normal_bf16(seed_seq: np.random.SeedSequence, shape, std: float) -> np.ndarray:
    """N(0, std^2) draws rounded to bf16, deterministic per (seed_seq, shape)."""
    n = int(np.prod(shape))
    nchunks = max(1, -(-n // CHUNK))
    kids = seed_seq.spawn(nchunks)
    out = np.empty(n, dtype=np.uint16)

    def fill(i):
        lo, hi = i * CHUNK, min(n, (i + 1) * CHUNK)
        g = np.random.Generator(np.random.PCG64(kids[i]))
        v = g.standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        out[lo:hi] = bf16_bits(v)

    if nchunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


def _streams(seed: int, names):
    kids = np.random.SeedSequence(seed).spawn(len(names))
    return dict(zip(names, kids))


def block_inputs(T, H, E, k, F, seed, zipf_s=None, zipf_scale=0.4, n_cold=0,
                 passages=None, passage_len=None, min_len=None, only=None, **_):
    """Inputs of the full block: x[T,H], w_r[H,E], w_gate/w_up[E,H,F],
    w_down[E,F,H], dy[T,H] (all bf16 bits) and mask[T] (uint8) or None.

    `only` (a set of names) skips the other expert-weight/gradient draws; every
    array is drawn from its own stream, so what is drawn does not change."""
    s = _streams(seed, ["x", "w_r", "w_gate", "w_up", "w_down", "dy", "aux"])

    def want(n):
        return only is None or n in only

    x = normal_bf16(s["x"], (T, H), 1.0)
    w_r = normal_bf16(s["w_r"], (H, E), WEIGHT_STD)
    w_gate = normal_bf16(s["w_gate"], (E, H, F), WEIGHT_STD) if want("w_gate") else None
    w_up = normal_bf16(s["w_up"], (E, H, F), WEIGHT_STD) if want("w_up") else None
    w_down = normal_bf16(s["w_down"], (E, F, H), WEIGHT_STD) if want("w_down") else None
    dy = normal_bf16(s["dy"], (T, H), 1.0) if want("dy") else None
    aux = np.random.Generator(np.random.PCG64(s["aux"]))
    mask = None
    if zipf_s is not None:
        # Popularity through the data: the last hidden channel is a constant 1
        # and its router row carries a per-expert bias proportional to the log
        # of a Zipf(s) popularity over a seeded expert permutation; the n_cold
        # least popular experts get a bias that keeps them unselected.
        perm = aux.permutation(E)
        rank = np.empty(E, dtype=np.int64)
        rank[perm] = np.arange(1, E + 1)
        logp = -zipf_s * np.log(rank.astype(np.float64))
        bias = (zipf_scale * logp).astype(np.float32)
        bias[rank > E - n_cold] = -1e4
        x[:, H - 1] = bf16_bits(np.ones(1, np.float32))[0]
        w_r[H - 1, :] = bf16_bits(bias)
    if passages is not None:
        lens = aux.integers(min_len, passage_len, size=passages, endpoint=True)
        pos = np.arange(passage_len)[None, :]
        mask = (pos < lens[:, None]).astype(np.uint8).reshape(-1)
        assert mask.size == T
    return dict(x=x, w_r=w_r, w_gate=w_gate, w_up=w_up, w_down=w_down, dy=dy,
                mask=mask, dims=dict(T=T, H=H, E=E, k=k, F=F))


EP_ROWS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tests", "golden", "ep_share_rows.json")


def ep_rows(T, H, E_total, k, seed, E):
    """Token index of each row a rank holding experts 0..E-1 receives, and
    the per-expert counts: the stored routing of the seed-`seed` batch (the
    file records the batch it was computed on)."""
    with open(EP_ROWS) as f:
        doc = json.load(f)
    src = doc["source"]
    want = dict(T=T, H=H, E=E_total, k=k, seed=seed, local_experts=E)
    if any(src[n] != v for n, v in want.items()):
        raise ValueError(f"{EP_ROWS} holds the routing of {src}, not {want}")
    return (np.asarray(doc["row_token"], dtype=np.int64),
            np.asarray(doc["counts"], dtype=np.int32))


def experts_inputs(H, E, F, seed, E_total, k, T, **_):
    """Inputs of one expert-parallel rank's share: xp[R,H] rows grouped
    expert-major, counts[E] (int32, sum R), w_gate/w_up[E,H,F], w_down[E,F,H],
    d_o[R,H].  The rows are the tokens of a T x H batch (drawn as the block
    workloads draw x, same seed) that a top-k router sends to experts 0..E-1,
    in expert-major, token-ascending order."""
    row_token, counts = ep_rows(T, H, E_total, k, seed, E)
    R = int(counts.sum())
    x = block_inputs(T=T, H=H, E=E_total, k=k, F=F, seed=seed, only=set())["x"]
    s = _streams(seed, ["xp", "counts", "w_gate", "w_up", "w_down", "d_o"])
    return dict(
        xp=np.ascontiguousarray(x[row_token]),
        counts=counts,
        w_gate=normal_bf16(s["w_gate"], (E, H, F), WEIGHT_STD),
        w_up=normal_bf16(s["w_up"], (E, H, F), WEIGHT_STD),
        w_down=normal_bf16(s["w_down"], (E, F, H), WEIGHT_STD),
        d_o=normal_bf16(s["d_o"], (R, H), 1.0),
        dims=dict(R=R, H=H, E=E, F=F))


def make(name: str, **overrides):
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    if cfg["kind"] == "experts":
        return experts_inputs(**cfg)
    return block_inputs(**cfg)
