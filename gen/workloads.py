"""The synthetic workloads, named by what they are.

Shapes follow the paper's training and retrieval setting: chunk size S=64
and top-k=8 (Experiments, Models), 12 heads of width 64 (Appendix A), and
context lengths from 16K to a 16M-token needle search (Experiments, Table 2).
Landmarks are one vector per chunk of width D = H*d, shared by all heads
(Eq. 1 scores one scalar per chunk pair), scaled by 1/sqrt(D).
"""

from dataclasses import dataclass, field
import math


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    S: int
    n_chunks: int          # causal: L/S ; decode: number of past chunks
    topk: int
    dtype: str             # "fp32" or "bf16"
    seed: int
    mode: str = "causal"   # "causal" or "decode"
    Hr: int = 1
    D: int = 0             # 0 -> H*d
    backward: bool = False
    planted: int = 0       # planted target chunks (long-range retrieval cases)
    margin: float = 1e-3   # k-th vs (k+1)-th landmark score gap enforced
    whole_reseed: bool = False   # redraw every input until all margins hold
    device_kv: bool = False      # K/V cache drawn on the device (too large for host)
    gumbel_seed: int = -1        # >= 0: Gumbel top-k selection with this generator seed
    lmk_row: bool = False        # query chunks carry their LMK token as an S+1-th row
    notes: str = field(default="", compare=False)

    @property
    def Dl(self) -> int:
        return self.D if self.D else self.H * self.d

    @property
    def n_query_chunks(self) -> int:
        return 1 if self.mode == "decode" else self.n_chunks

    @property
    def Sq(self) -> int:
        """Query rows per chunk: S, or S + 1 with the LMK row."""
        return self.S + 1 if self.lmk_row else self.S

    @property
    def Lq(self) -> int:
        return self.n_query_chunks * self.Sq

    @property
    def Lkv(self) -> int:
        return self.n_chunks * self.S

    @property
    def score_scale(self) -> float:
        return 1.0 / math.sqrt(self.Dl)

    @property
    def attn_scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def tokens(self) -> int:
        """Query tokens processed by one pass of the path."""
        return self.B * self.Lq


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny_fp32_1k", B=1, H=1, d=64, S=64, n_chunks=16, topk=2,
                 dtype="fp32", seed=1, whole_reseed=True,
                 notes="1,024 tokens, 16 chunks, fp32"),
        Workload("train_16k_bf16", B=8, H=12, d=64, S=64, n_chunks=256, topk=8,
                 dtype="bf16", seed=2,
                 notes="16,384 tokens, width 768, 256 chunks"),
        Workload("fwdbwd_64k_bf16", B=2, H=16, d=64, S=64, n_chunks=1024, topk=8,
                 dtype="bf16", seed=3, backward=True,
                 notes="65,536 tokens, forward and backward"),
        Workload("planted_1m_bf16", B=1, H=8, d=64, S=64, n_chunks=16384, topk=8,
                 dtype="bf16", seed=4, planted=8,
                 notes="1,048,576 tokens, eight planted targets for the last chunk"),
        Workload("decode_16m_bf16", B=1, H=8, d=64, S=64, n_chunks=262144, topk=8,
                 dtype="bf16", seed=5, mode="decode", planted=1, device_kv=True,
                 notes="one new chunk against 16,777,216 cached tokens"),
    ]
}


def get_workload(name: str, **overrides) -> Workload:
    """Look up a workload; keyword overrides give reduced or varied shapes."""
    w = WORKLOADS[name]
    if overrides:
        fields = dict(w.__dict__)
        fields.update(overrides)
        w = Workload(**fields)
    return w
