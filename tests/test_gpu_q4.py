"""GPU parity of the Q4_0 stack at full size (30 layers, hidden 2816, 128 experts,
top-8, intermediate 1408, 45 slots, 96 tokens), as in the A3B full-size test."""
import pytest

import synth
from gpu_common import store_buffer
from test_gpu_full import verify_chain

pytestmark = pytest.mark.gpu


def test_q4_decode_full_size():
    wl = synth.WORKLOADS["q4_decode"]
    st = store_buffer(wl)
    try:
        verify_chain(wl, wl.budget_slots, wl.rho, st, 16, 4)
    finally:
        st[0].free()
