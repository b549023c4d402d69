"""The five synthetic workloads: corpus recipe, query recipe and search knobs.

They stand in for the paper's ColBERTv2-embedded LoTTE, HotpotQA and
MS MARCO collections (Sec. 5.1, Table 1), which are not available here: 128-d
unit vectors on the grid G, clustered (noise sigma 0.05) around random unit
centroids, with queries that are noised (sigma 0.1) copies of a random
document's tokens.  ``8.8m`` has MS MARCO's shape (8.8M docs, ~600M tokens).
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    ndocs: int
    ncent: int
    nbits: int
    nq: int
    Tq: int
    nprobe: int
    ncand: int
    k: int
    len_kind: int          # 0 fixed, 1 lognormal, 2 uniform
    len_lo: int
    len_hi: int
    len_mean: float = 0.0
    pop_kind: int = 0      # 0 uniform, 1 zipf
    zipf_s: float = 1.1
    q_dtype: str = "bf16"  # storage type of the query tensor handed to the search
    dim: int = 128
    tok_sigma: float = 0.05
    q_sigma: float = 0.1
    len_sigma: float = 0.5
    notes: str = field(default="", compare=False)

    def corpus_spec(self):
        from . import CorpusSpec
        return CorpusSpec(seed=self.seed, ndocs=self.ndocs, ncent=self.ncent, dim=self.dim,
                          len_kind=self.len_kind, len_lo=self.len_lo, len_hi=self.len_hi,
                          len_mean=self.len_mean, len_sigma=self.len_sigma, pop_kind=self.pop_kind,
                          zipf_s=self.zipf_s, tok_sigma=self.tok_sigma, q_sigma=self.q_sigma)

    def scaled(self, **kw) -> "Workload":
        d = self.__dict__.copy()
        d.update(kw)
        return Workload(**d)


WORKLOADS = {
    "tiny": Workload("tiny", seed=1001, ndocs=1000, ncent=1024, nbits=2, nq=16, Tq=32,
                     nprobe=2, ncand=256, k=10, len_kind=0, len_lo=32, len_hi=32, q_dtype="f32"),
    "100k": Workload("100k", seed=1002, ndocs=100_000, ncent=16_384, nbits=2, nq=256, Tq=32,
                     nprobe=4, ncand=4096, k=10, len_kind=1, len_lo=8, len_hi=180, len_mean=64.0),
    "1m": Workload("1m", seed=1003, ndocs=1_000_000, ncent=65_536, nbits=2, nq=1024, Tq=32,
                   nprobe=8, ncand=8192, k=100, len_kind=1, len_lo=8, len_hi=180, len_mean=70.0,
                   pop_kind=1),
    "8.8m": Workload("8.8m", seed=1004, ndocs=8_800_000, ncent=262_144, nbits=2, nq=4096, Tq=32,
                     nprobe=16, ncand=16_384, k=100, len_kind=1, len_lo=8, len_hi=180, len_mean=70.0,
                     pop_kind=1),
    "2m-long": Workload("2m-long", seed=1005, ndocs=2_000_000, ncent=65_536, nbits=4, nq=512, Tq=64,
                        nprobe=32, ncand=32_768, k=1000, len_kind=2, len_lo=128, len_hi=512),
}
