"""Parity at the Vicuna-33B shape (Table 1: 60 layers, d 6656, 52 heads of
128; F 17920, V 32000, bf16, 4 draft heads, 64-node tree) through
properties that hold at any size: on the 512-token workload with forced
acceptance p = 0.7 the speculative stream equals the GPU's greedy stream
token for token and every step accepts exactly 1 + (consecutive seeded
successes) tokens along the rank-0 chain."""
import pytest

import synth
from gpu_helpers import forced_lossless_run, log

pytestmark = pytest.mark.gpu


def test_vicuna33b_lossless_and_forced_acceptance():
    log("vicuna33b: generating weights on the GPU")
    w = synth.make_weights(synth.VICUNA33B, device="cuda")
    forced_lossless_run(synth.VICUNA33B, w, synth.WORKLOADS["vicuna33b_p512"], steps=12)
