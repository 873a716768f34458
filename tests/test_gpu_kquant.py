"""GPU parity of the K-quant formats (Q4_K, Q6_K and the Q4_K_M mix: Q4_K gate/up, Q6_K down)
through the C ABI: the decode GEMVs over super-blocks against the exact oracle, in every
copy mode, on several shapes, on stores tiled with the hand-worked super-blocks of
tests/golden/kquant_hand_blocks.txt (signed, subnormal and zero scales, 6-bit packing
extremes), and on the A3B-topology Q4_K_M stack at full size (48 layers, 35 % cache)."""
import pytest

import synth
from edge_blocks import edge_tokens, kquant_golden_store
from gpu_common import store_buffer
from test_gpu_decode import run_decode
from test_gpu_full import verify_chain
from test_gpu_prefill import run_prefill

pytestmark = pytest.mark.gpu


def kq_workload(qtype, **kw):
    base = dict(qtype=qtype, n_layers=2, hidden=512, inter=256, n_experts=16, top_k=4,
                name=f"kq_{qtype}")
    base.update(kw)
    return synth.WORKLOADS["tiny"].with_(**base)


@pytest.mark.parametrize("qtype", ["q4_k_m", "q4_k", "q6_k"])
def test_kquant_decode_copy_modes(qtype):
    wl = kq_workload(qtype)
    store = store_buffer(wl)
    for mode in ("kernel", "split", "side", "sdma"):
        run_decode(wl, 6, residual=True, prenorm=True, n_tokens=10, store=store,
                   copy_mode=mode)[0].close()
    run_decode(wl, 6, n_tokens=8, store=store)[0].close()
    store[0].free()


@pytest.mark.parametrize("shape", [(256, 256, 8, 2, 2), (2048, 768, 32, 8, 9), (1024, 512, 64, 6, 7),
                                   (768, 1280, 16, 8, 8), (4096, 256, 16, 16, 16),
                                   (256, 3072, 4, 4, 4), (1024, 768, 256, 16, 20)])
@pytest.mark.parametrize("qtype", ["q4_k_m", "q4_k", "q6_k"])
def test_kquant_decode_shapes(qtype, shape):
    H, I, E, k, C = shape
    wl = kq_workload(qtype, hidden=H, inter=I, n_experts=E, top_k=k, name=f"kq{H}x{I}x{E}")
    run_decode(wl, C, residual=True, prenorm=True, n_tokens=5)[0].close()


@pytest.mark.parametrize("qtype", ["q4_k_m", "q4_k", "q6_k"])
def test_kquant_hand_worked_super_blocks(qtype):
    """Every super-block a hand-worked one: signed d, dmin and scales, subnormal d, 6-bit
    scale/min packing extremes; tokens with an all-zero row and a 1e-6 .. 1e3 row."""
    wl = kq_workload(qtype)
    keep, ptr, arr = store_buffer(wl)
    kquant_golden_store(arr, wl)
    X = edge_tokens(synth.hidden(wl, n_tokens=8))
    for prenorm, residual in ((False, False), (True, False), (True, True)):
        run_decode(wl, 6, residual=residual, prenorm=prenorm, n_tokens=8, store=(keep, ptr, arr),
                   X=X)[0].close()
    keep.free()


def test_q4km_decode_full_size():
    wl = synth.WORKLOADS["q4km_decode"]
    st = store_buffer(wl)
    try:
        verify_chain(wl, wl.budget_slots, wl.rho, st, 16, 6)
    finally:
        st[0].free()


@pytest.mark.parametrize("qtype", ["q4_k_m", "q4_k", "q6_k"])
def test_kquant_prefill_and_small_calls(qtype):
    """Multi-token calls: 300 tokens with 6 slots (the MFMA grouped GEMMs on bf16 tiles
    dequantised from the super-blocks, slots reused inside the call), 5 tokens whose experts
    fit (the decode GEMVs per token) and 8 tokens with 5 slots (the host-table path, MFMA)."""
    wl = kq_workload(qtype, hidden=1024, inter=512)
    store = store_buffer(wl)
    run_prefill(wl, 6, 300, calls=2, prenorm=True, residual=True, store=store)
    run_prefill(wl, 16, 5, calls=2, prenorm=True, residual=True, store=store)
    run_prefill(wl, 5, 8, calls=2, prenorm=True, residual=True, store=store)
    store[0].free()


@pytest.mark.parametrize("qtype", ["q4_k_m", "q6_k"])
def test_kquant_prefill_rows_past_first_tile(qtype):
    """2048 tokens, 16 experts, top-2: about 256 rows per expert, a full 256-row tile and a
    partial second one for many experts; every token's y compared, hand-worked super-blocks."""
    wl = kq_workload(qtype, n_layers=1, hidden=1024, inter=512, top_k=2)
    keep, ptr, arr = store_buffer(wl)
    kquant_golden_store(arr, wl, seed=3)
    xs = [synth.hidden(wl.with_(hidden_seed=91), rho=-1.0, n_tokens=2048)]
    run_prefill(wl, 6, 2048, calls=1, prenorm=True, residual=False, store=(keep, ptr, arr), xs=xs)
    keep.free()
