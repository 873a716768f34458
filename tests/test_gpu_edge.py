"""GPU parity on the corners of the block formats and of the inputs, through the C ABI.

Stores rewritten by ``edge_blocks.edge_store`` (negative, subnormal and zero fp16 scales,
Q8_0 bytes -128 / +127, Q4_0 nibbles 0 / 15, signed-extreme Q4_0 scales, the hand-worked
blocks of ``tests/golden/quant_hand_blocks.txt``), hidden states with an all-zero token and
a token whose 32-wide blocks span 1e-6 .. 1e3, run through decode (copy kernel fused with
gate/up, split launches, copy engine on a side stream), small multi-token calls (union fits
the slots / exceeds them) and the bf16 MFMA prefill.  Every call is compared with the
oracle (exact oracle for the GEMV paths, bf16-weight oracle for the MFMA GEMMs): routes,
trace and counters exact, y within 2e-3 x RMS.

Also here: a prefill call with about 256 rows per expert (a second, partial 128-row tile
of every expert's GEMMs) compared on every row, and slots poisoned with 0xFF bytes before
use (every slot scale reads NaN until the expert is copied in), so that a read of a slot
before its copy has landed would show up as a non-finite output.
"""
import pytest

import synth
from edge_blocks import REGIMES, edge_store, edge_tokens
from gpu_common import log, store_buffer
from test_gpu_decode import run_decode
from test_gpu_prefill import run_prefill

pytestmark = pytest.mark.gpu


def edge_workload(qtype, **kw):
    base = dict(qtype=qtype, n_layers=2, hidden=512, inter=256, n_experts=16, top_k=4,
                name=f"edge_{qtype}")
    base.update(kw)
    return synth.WORKLOADS["tiny"].with_(**base)


def edge_buffer(wl, regime, seed=0):
    keep, ptr, arr = store_buffer(wl)
    edge_store(arr, wl, regime, seed)
    log(f"  store rewritten: regime {regime}")
    return keep, ptr, arr


@pytest.mark.parametrize("regime", REGIMES)
@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_edge_blocks_decode(qtype, regime):
    wl = edge_workload(qtype)
    store = edge_buffer(wl, regime)
    X = edge_tokens(synth.hidden(wl, n_tokens=10))
    # (the residual variant: y = fp32(x + moe), so where the MoE output is far below the
    # residual's ulp -- subnormal scales -- only the variants without it see its error)
    for mode in ("kernel", "split", "side"):
        for prenorm, residual in ((False, False), (True, False), (True, True)):
            run_decode(wl, 6, residual=residual, prenorm=prenorm, n_tokens=10, store=store,
                       copy_mode=mode, X=X)[0].close()
    store[0].free()


@pytest.mark.parametrize("regime", REGIMES)
@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_edge_blocks_small_calls(qtype, regime):
    """5 tokens whose experts fit 16 slots (union GEMVs, table on the device) and 8 tokens
    with 5 slots (host-table path, slots reused inside the call)."""
    wl = edge_workload(qtype)
    store = edge_buffer(wl, regime)
    for T, budget in ((5, 16), (8, 5)):
        xs = [edge_tokens(synth.hidden(wl.with_(hidden_seed=40 + c), rho=-1.0, n_tokens=T),
                          seed=c) for c in range(2)]
        for residual in (False, True):
            run_prefill(wl, budget, T, calls=2, prenorm=True, residual=residual, store=store,
                        xs=xs)
    store[0].free()


@pytest.mark.parametrize("regime", REGIMES)
@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_edge_blocks_prefill(qtype, regime):
    """The bf16 MFMA grouped GEMMs (every route, y of every token) on 160 tokens with 6 slots
    (slots reused inside the call), with and without the pre-norm."""
    wl = edge_workload(qtype, hidden=1024, inter=384)
    store = edge_buffer(wl, regime)
    xs = [edge_tokens(synth.hidden(wl.with_(hidden_seed=60), rho=-1.0, n_tokens=160))]
    for prenorm, residual in ((False, False), (True, False), (True, True)):
        run_prefill(wl, 6, 160, calls=1, prenorm=prenorm, residual=residual, store=store, xs=xs)
    store[0].free()


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_prefill_rows_past_first_tile(qtype):
    """2048 tokens over 16 experts, top-2: about 256 rows per expert, so every expert's
    GEMMs run a full 128-row tile and a partial second (or third) one; y of every token is
    compared, with 6 slots (waves of slot reuse) and with every expert resident."""
    wl = edge_workload(qtype, n_layers=1, hidden=1024, inter=384, top_k=2)
    store = store_buffer(wl)
    xs = [synth.hidden(wl.with_(hidden_seed=90), rho=-1.0, n_tokens=2048)]
    for budget in (6, 16):
        run_prefill(wl, budget, 2048, calls=1, prenorm=True, residual=True, store=store, xs=xs)
    store[0].free()


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_poisoned_slots(qtype):
    """Slots filled with 0xFF bytes before the first call (each slot scale is then a NaN
    until its expert is copied in): decode in the copy modes, small calls and prefill with
    slot reuse inside a call stay finite and equal to the oracle."""
    wl = edge_workload(qtype, hidden=1024, inter=384)
    store = store_buffer(wl)
    for mode in ("kernel", "split", "side", "sdma"):
        run_decode(wl, 5, residual=True, prenorm=True, n_tokens=8, store=store, copy_mode=mode,
                   poison=True)[0].close()
    for T, budget in ((5, 16), (8, 5), (300, 6)):
        for mode in ("kernel", "side"):
            run_prefill(wl, budget, T, calls=2, prenorm=True, residual=True, store=store,
                        copy_mode=mode, poison=True)
    store[0].free()
