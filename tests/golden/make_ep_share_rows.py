"""Writes ep_share_rows.json: the rows one expert-parallel rank receives.

The ep_share workload is the local expert FFN of one rank under expert
parallelism (paper §3, "Expert parallelism and topology": experts are split
over the ranks and each rank runs its own experts on the token rows routed to
them).  Its rows are those a top-8-of-128 router sends to experts 0..15 (the
rank that holds the first 16 experts) on a T=8192, H=2048 batch drawn like the
Qwen-shape workload with seed 2.  The routing is the oracle's: logits, top-k
selection and the expert-major, token-ascending permutation.  Only the oracle
is called; the stored token indices and counts are its output.

    python tests/golden/make_ep_share_rows.py
"""
from __future__ import annotations

import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402
from oracle import moe_oracle as o  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ep_share_rows.json")
SOURCE = dict(T=8192, H=2048, E=128, k=8, seed=2, local_experts=16)


def compute():
    s = SOURCE
    inp = workloads.block_inputs(T=s["T"], H=s["H"], E=s["E"], k=s["k"], F=128, seed=s["seed"], only=set())
    z = o.router_logits(o.widen_bf16(inp["x"]), o.widen_bf16(inp["w_r"]))
    idx = o.select_topk(z, s["k"])
    counts, offsets, row_token, _ = o.permutation(idx, s["E"])
    n = s["local_experts"]
    return [int(c) for c in counts[:n]], [int(t) for t in row_token[:offsets[n]]]


def main():
    counts, row_token = compute()
    doc = {
        "what": "Token index of each row routed to experts 0..15 (expert-major, tokens ascending within an "
                "expert) and the per-expert row counts, from the oracle router on the seed-2 Qwen-shape batch.",
        "cite": "Paper §3, 'Expert parallelism and topology': one rank's experts run on the rows routed to them.",
        "source": SOURCE,
        "counts": counts,
        "row_token": row_token,
    }
    with open(OUT, "w") as f:
        json.dump(doc, f, separators=(",", ":"))
        f.write("\n")
    print(f"wrote {OUT}: {len(row_token)} rows over {len(counts)} experts")


if __name__ == "__main__":
    main()
