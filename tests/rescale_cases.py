"""Inputs on which the kernels' lazy running max must move after the first
tile (the rescale of a non-zero accumulator), shared by the GPU parity tests
and the CPU check that these inputs really take that path.

With N(0, 1) inputs and the default scale 1/sqrt(d) a row's max is set on
its first tile and never passes the 2^13 sum limit later, so the parity
cases use ``softmax_scale = 1.0`` (logits sqrt(d) times wider) and, in one
case, a key planted late in the sequence along a query.  That key's logit
sits about 40 base-2 units above the rest of its row at the default scale
(a finite stale probability near 2^40) and about 460 at scale 1.0, where the
probabilities taken against the stale max overflow to +inf and the sum
check has to catch an infinite sum, not just a large one.
"""
import dataclasses

import numpy as np

from paper_2502_12085_amd import inputs

SCALE = 1.0

# name -> problem (n_hosts, host_idx, La, Lb, l_p, n_q, n_kv, d)
ATTENTION = {
    "tiny_d64": inputs.WORKLOADS["tiny"].problem,
    "ragged_d128": inputs.Problem(4, 2, 100, 333, 17, 6, 2, 128),
    "d64_mid": inputs.Problem(4, 3, 512, 2048, 250, 8, 2, 64),
    "ragged_d128_planted": inputs.Problem(4, 2, 100, 333, 17, 6, 2, 128),
}

# the planted key: local key PLANT_KEY of KV head 0 is 3x the query of query
# head 0 at row PLANT_ROW (a local row that sees it, 3 tiles in)
PLANT_ROW = 400
PLANT_KEY = 290


def attention_inputs(name):
    p = ATTENTION[name]
    inp = inputs.make_inputs(inputs.Workload(name, p), seed=77)
    if name.endswith("_planted"):
        q = inputs.bf16_bits_to_f32(inp["q"][0, PLANT_ROW])
        k = inp["k"].copy()
        k[0, p.anchor_len + PLANT_KEY] = inputs.f32_to_bf16_bits(q * np.float32(3.0))
        inp["k"] = k
    return p, inp


# decode shapes (n_q, n_kv, d, Lc, n_new, append) whose split plan is one
# split, so that the emulation of the block walk applies: the one-wave kernel
# (32-key blocks, 3 of them) and the eight-wave kernel (128-key tiles, 3 of
# them, two 256-row groups); plus a many-split one-wave shape
DECODE_ONE_SPLIT = {
    "one_wave": ((8, 2, 128, 90, 1, 1), 32),
    "eight_wave": ((16, 2, 128, 300, 40, 1), 128),
}
DECODE_MANY_SPLITS = (8, 2, 128, 1000, 1, 1)


def decode_inputs(shape, seed=78):
    n_q, n_kv, d, lc, n_new, app = shape
    case = inputs.make_decode_case(n_q, n_kv, d, [lc], n_new, seed=seed)
    kc, vc = case["caches"][0]
    return case["q"], kc, vc, (case["k_new"] if app else None), (case["v_new"] if app else None)


def with_host(p, host_idx):
    return dataclasses.replace(p, host_idx=host_idx)
