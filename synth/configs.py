"""The synthetic workloads of the expert-slot-cache MoE FFN, by name.

Shapes stand in for the paper's GGUF model profiles (its model-profile
table): an "A3B"-shaped Q8_0 stack, a Q4_0 stack and a tiny one-layer case.
Nothing here computes anything of the method; it only names sizes, seeds and
distributions for the generator in this package.
"""
from dataclasses import dataclass, field, replace
from typing import Tuple

# format name -> (bytes per block, weights per block, type code)
FORMATS = {"q8_0": (34, 32, 8), "q4_0": (18, 32, 2), "q4_k": (144, 256, 12), "q6_k": (210, 256, 14)}
# a model type naming a mix: (gate/up format, down format)
MIXES = {"q4_k_m": ("q4_k", "q6_k")}


@dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    hidden: int
    n_experts: int
    top_k: int
    inter: int
    qtype: str                 # "q8_0", "q4_0", "q4_k", "q6_k" or "q4_k_m" (Q4_K gate/up, Q6_K down)
    weight_sigma: float        # expert weights ~ N(0, sigma) before quantisation
    router_sigma: float        # router W_r ~ N(0, sigma), fp32 [hidden, n_experts]
    n_tokens: int              # decode: tokens generated one at a time; prefill: chunk size
    rho: float                 # AR(1) coefficient of the hidden-state drift; <0 means iid N(0,1)
    budget_slots: int          # expert slots per layer
    model_seed: int            # seed of the expert store and routers
    hidden_seed: int           # seed of the hidden states
    mode: str = "decode"       # "decode" (one token per layer call) or "prefill" (whole chunk per call)
    sweep_slots: Tuple[int, ...] = field(default=())
    sweep_rhos: Tuple[float, ...] = field(default=())
    cache_percent: float = 0.0  # the cache budget as a percentage of each layer's experts
    horizon: int = 0            # verify mode: draft tokens per verification window (window = 1 + horizon)
    accept_q: float = 0.0       # verify mode: probability that a draft token passes verification

    @property
    def formats(self) -> Tuple[str, str]:
        """(gate/up format, down format)."""
        return MIXES.get(self.qtype, (self.qtype, self.qtype))

    @property
    def block_bytes(self) -> int:
        """Bytes per block of the gate/up format (Q8_0 / Q4_0 workloads: every matrix)."""
        return FORMATS[self.formats[0]][0]

    @property
    def qcode(self) -> int:
        """Type code used by the C interfaces: the gate/up format's code (8 Q8_0, 2 Q4_0,
        12 Q4_K, 14 Q6_K), with the down format's code in the next byte when it differs."""
        gu, dn = self.formats
        return FORMATS[gu][2] | (0 if dn == gu else FORMATS[dn][2] << 8)

    @property
    def matrix_bytes(self) -> int:
        """Bytes of one gate (or up) matrix."""
        bb, wpb, _ = FORMATS[self.formats[0]]
        return self.inter * self.hidden // wpb * bb

    @property
    def down_bytes(self) -> int:
        bb, wpb, _ = FORMATS[self.formats[1]]
        return self.inter * self.hidden // wpb * bb

    @property
    def payload_bytes(self) -> int:
        return 2 * self.matrix_bytes + self.down_bytes

    @property
    def store_bytes(self) -> int:
        return self.n_layers * self.n_experts * self.payload_bytes

    def hidden_stream(self, rho: float) -> int:
        """Stream id of the hidden states for a given rho (iid when rho < 0)."""
        return 255 if rho < 0 else int(round(10 * rho))

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Workload("tiny", n_layers=1, hidden=256, n_experts=16, top_k=2, inter=128,
                qtype="q8_0", weight_sigma=0.02, router_sigma=0.1, n_tokens=64, rho=0.8,
                budget_slots=4, model_seed=1, hidden_seed=1, cache_percent=25)

A3B_DECODE = Workload("a3b_decode", n_layers=48, hidden=2048, n_experts=128, top_k=8, inter=768,
                      qtype="q8_0", weight_sigma=0.02, router_sigma=0.05, n_tokens=96, rho=0.8,
                      budget_slots=19, model_seed=2, hidden_seed=2, cache_percent=15)

A3B_SWEEP = A3B_DECODE.with_(name="a3b_sweep", hidden_seed=3, sweep_slots=(19, 45, 96),
                             sweep_rhos=(0.3, 0.9))

Q4_DECODE = Workload("q4_decode", n_layers=30, hidden=2816, n_experts=128, top_k=8, inter=1408,
                     qtype="q4_0", weight_sigma=0.02, router_sigma=0.05, n_tokens=96, rho=0.8,
                     budget_slots=45, model_seed=4, hidden_seed=4, cache_percent=35)

# The paper's 4-bit profile is Q4_K_M of the same A3B topology: Q4_K gate and up, Q6_K down
# (hidden 2048 and intermediate 768 are multiples of the 256-weight super-block).  Same
# weights' distribution and hidden-state stream as a3b_decode; 35 % cache (45 slots).
A3B_Q4KM_DECODE = A3B_DECODE.with_(name="q4km_decode", qtype="q4_k_m", budget_slots=45,
                                   cache_percent=35, model_seed=6, hidden_seed=2)

A3B_PREFILL = A3B_DECODE.with_(name="a3b_prefill", n_tokens=4096, rho=-1.0, budget_slots=45,
                               cache_percent=35,
                               hidden_seed=5, mode="prefill")

# Prefill of the Q4_K_M A3B stack (Q4_K gate/up, Q6_K down): the K-quant grouped GEMMs.
A3B_Q4KM_PREFILL = A3B_PREFILL.with_(name="q4km_prefill", qtype="q4_k_m", model_seed=6)

# Speculative verification windows through the A3B stack: 1 + 4 tokens per layer call, each
# draft accepted with probability 0.75 until the first rejection; 25 % cache (32 slots), the
# paper's setting for its speculative comparison.  Same weights and hidden-state stream as
# a3b_decode (the first 96 states are the decode workload's).
A3B_VERIFY = A3B_DECODE.with_(name="a3b_verify", budget_slots=32, cache_percent=25, horizon=4,
                              accept_q=0.75, mode="verify")

WORKLOADS = {w.name: w for w in (TINY, A3B_DECODE, A3B_SWEEP, Q4_DECODE, A3B_Q4KM_DECODE, A3B_PREFILL,
                                 A3B_Q4KM_PREFILL, A3B_VERIFY)}
