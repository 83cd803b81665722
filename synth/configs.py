"""The workload shapes of the lifelong-sequence NN-select + encode path.

Each shape follows the paper's scales: a lifelong sequence of O(10^4) actions
(Sec. 3.2.2, after Eq. 3), a selected sequence of O(10^2) tokens, and thousands
of candidate items per ranking request (Sec. 1).  The encoder sizes are fixed
per workload; the paper's own production encoder (d_model 64 / 1 head / FFN 32 /
2 layers of Sec. 3.2.2) is the paper workload's.

This module holds shapes only: no arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    cid: int                      # 1..5, also the data seed
    name: str
    dtype: str                    # "f32" or "bf16": storage and MFMA operand type; "i8":
                                  # int8 sequence codes, bf16 candidates (NN search only)
    R: int                        # requests (users) in one batch
    L: Optional[int]              # lifelong length per request (fixed), or None
    L_range: Optional[Tuple[int, int]]  # inclusive [lo, hi] when ragged
    d: int                        # embedding width of actions and candidates
    N: int                        # candidates per request
    k: int                        # NN top-k over the lifelong sequence
    d_model: int
    n_heads: int
    d_ffn: int
    n_layers: int
    has_time: bool                # time-bucket feature present
    rt_len: int = 0               # real-time actions per request
    tie_frac: float = 0.0         # fraction of rows overwritten with another row's embedding
    # Eq. 2's other sources: rt_keep of the real-time rows kept as they are (-1: all
    # of them), an NN top-k_rt over the rest, and an NN top-k_imp over an
    # impression sequence of imp_len rows
    rt_keep: int = -1
    k_rt: int = 0
    imp_len: int = 0
    k_imp: int = 0
    encode: bool = True           # the encoder follows the NN search

    @property
    def r(self) -> int:
        """Real-time rows kept unconditionally (S_RT[:r] of Eq. 2)."""
        return self.rt_len if self.rt_keep < 0 else self.rt_keep

    @property
    def T(self) -> int:
        """Encoder positions: the k NN tokens, the kept real-time rows and the NN
        tokens of the real-time rest and of the impressions."""
        return self.k + self.r + self.k_rt + self.k_imp

    @property
    def total_candidates(self) -> int:
        return self.R * self.N

    @property
    def data_seed(self) -> int:
        return self.cid

    @property
    def weight_seed(self) -> int:
        return 100 + self.cid


TINY = Workload(1, "tiny_f32", "f32", R=1, L=1024, L_range=None, d=64, N=16, k=32,
                d_model=64, n_heads=2, d_ffn=128, n_layers=1, has_time=False)
SINGLE = Workload(2, "single_bf16", "bf16", R=1, L=16384, L_range=None, d=256, N=1000,
                  k=256, d_model=256, n_heads=4, d_ffn=1024, n_layers=2, has_time=True)
RAGGED = Workload(3, "ragged_bf16", "bf16", R=64, L=None, L_range=(1024, 16384), d=256,
                  N=500, k=128, d_model=256, n_heads=4, d_ffn=512, n_layers=2, has_time=True)
MIXED = Workload(4, "mixed_bf16", "bf16", R=1, L=16384, L_range=None, d=256, N=1000,
                 k=256, d_model=256, n_heads=4, d_ffn=1024, n_layers=2, has_time=True,
                 rt_len=100)
STRESS = Workload(5, "stress_bf16", "bf16", R=16, L=16384, L_range=None, d=256, N=4000,
                  k=512, d_model=256, n_heads=8, d_ffn=1024, n_layers=2, has_time=True,
                  tie_frac=0.01)

WORKLOADS = {w.cid: w for w in (TINY, SINGLE, RAGGED, MIXED, STRESS)}
# NN search over the paper's int8 sequence storage (32-d codes, Sec. 3.2.1) with
# dequantisation and L2 normalisation fused into the score kernel (Sec. 3.4.2);
# one request of the single workload's size.  The encoder fields are unused.
SELECT_I8 = Workload(6, "select_i8", "i8", R=1, L=16384, L_range=None, d=32, N=1000, k=256,
                     d_model=256, n_heads=4, d_ffn=1024, n_layers=2, has_time=True,
                     tie_frac=0.01, encode=False)
# The whole of Eq. 2 (Sec. 3.2.2): NN(S_LL, c) + S_RT[:r] + NN(S_RT[r:], c) +
# NN(S_imp, c), with real-time and impression sequences of O(10^2) actions; the
# single workload's lifelong sequence, candidates and encoder.
EQ2 = Workload(7, "eq2_bf16", "bf16", R=1, L=16384, L_range=None, d=256, N=1000, k=256,
               d_model=256, n_heads=4, d_ffn=1024, n_layers=2, has_time=True, rt_len=200,
               rt_keep=32, k_rt=32, imp_len=300, k_imp=64)
# The paper's production encoder (Sec. 3.2.2: d_model 64, one head, FFN 32, two
# layers; Sec. 4.4.2: 192 positions) on its 32-d PinSage embeddings (Sec. 3.2.1),
# for a batch of 256 candidates (the production batch of Sec. 4.4.3); the 192
# positions are the top-128 NN tokens and 64 real-time actions.
PAPER = Workload(8, "paper_bf16", "bf16", R=1, L=16384, L_range=None, d=32, N=256, k=128,
                 d_model=64, n_heads=1, d_ffn=32, n_layers=2, has_time=True, rt_len=64)
# The paper's production path end to end: the lifelong and real-time sequences
# stored as 32-d int8 codes (Sec. 3.2.1), the NN search with fused dequantisation
# and L2 normalisation (Sec. 3.4.2), and the production encoder on the
# dequantised rows.
PAPER_I8 = Workload(9, "paper_i8", "i8", R=1, L=16384, L_range=None, d=32, N=256, k=128,
                    d_model=64, n_heads=1, d_ffn=32, n_layers=2, has_time=True, rt_len=64)
BY_NAME = {w.name: w for w in list(WORKLOADS.values()) + [SELECT_I8, EQ2, PAPER, PAPER_I8]}


def scaled(w: Workload, **changes) -> Workload:
    """A copy of `w` with some fields replaced (small parity cases)."""
    from dataclasses import replace
    return replace(w, **changes)
