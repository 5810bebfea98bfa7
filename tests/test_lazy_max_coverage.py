"""The rescale parity cases really exercise the kernels' late max raise.

Replays, on the CPU, the lazy running-max decision of the prefill and decode
kernels (``lazy_max_emulation``) on the exact inputs of the GPU parity cases
in ``rescale_cases`` and checks that the branch which rescales a non-zero
accumulator runs after the first tile, while on the default scale it does
not (which is why those cases exist).  No GPU needed.
"""
import pytest

import lazy_max_emulation as emu
import rescale_cases as rc
from paper_2502_12085_amd import apb


@pytest.mark.parametrize("name", list(rc.ATTENTION))
def test_attention_cases_raise_the_max_after_the_first_tile(name):
    p, inp = rc.attention_inputs(name)
    n = emu.prefill_late_raises(inp["q"], inp["k"], inp["v"], inp["k_pass"], p.anchor_len,
                                scale=rc.SCALE)
    assert n >= 3, (name, n)


def test_planted_key_raises_its_wave_late():
    p, inp = rc.attention_inputs("ragged_d128_planted")
    # query head 0 alone: default scale; the planted key still forces a raise
    n = emu.prefill_late_raises(inp["q"], inp["k"], inp["v"], inp["k_pass"], p.anchor_len,
                                heads=[0])
    assert n >= 1
    _, clean = rc.attention_inputs("ragged_d128")
    assert emu.prefill_late_raises(clean["q"], clean["k"], clean["v"], clean["k_pass"],
                                   p.anchor_len, heads=[0]) == 0


def test_default_scale_never_raises_late_on_these_inputs():
    p, inp = rc.attention_inputs("tiny_d64")
    assert emu.prefill_late_raises(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                   p.anchor_len) == 0


@pytest.mark.parametrize("name", list(rc.DECODE_ONE_SPLIT))
def test_decode_cases_raise_the_max_after_the_first_block(name):
    shape, block = rc.DECODE_ONE_SPLIT[name]
    n_q, n_kv, d, lc, n_new, app = shape
    # the emulation walks one split: the library's plan must be one split
    # (a partial per row: fp32 O and LSE, or on the eight-wave path for 128
    # or more rows per KV head fp16 O, its scale and the LSE)
    ws = apb.decode_workspace_size(apb.DecodeProblem(*shape))
    per_row = 2 * d + 8 if (n_q // n_kv) * n_new >= 128 else (d + 1) * 4
    assert ws == n_q * n_new * per_row
    q, kc, _, kn, _ = rc.decode_inputs(shape)
    assert emu.decode_late_raises(q, kc, kn, block, scale=rc.SCALE) >= 1
    assert emu.decode_late_raises(q, kc, kn, block) == 0
