"""The five synthetic ct x pt linear-layer workloads.

Shapes stand in for the paper's models (GPT-2-124M and Qwen3-0.6B projection
and FFN layers, section 5.1); no checkpoint or dataset is used.  Weights are
drawn N(0, 0.02^2) as a stand-in for trained weights.

c1  tiny end-to-end case: N=2^10, 2 limbs, scale 2^25, 16 -> 16, activations
    encoded and encrypted, scalar weights, MAC + one rescale, decrypted.
c2  GPT-2-124M attention output projection: N=2^14, 4 limbs, 2^26, 768 -> 768.
c3  GPT-2-124M FFN up projection: N=2^15, 6 limbs, 2^26, 768 -> 3072, plus a
    standalone NTT/INTT over all 3072*2*6 output polynomials.
c4  Qwen3-0.6B gate+up projections stacked: N=2^16, 8 limbs, 2^28, 1024 -> 6144.
c5  full-polynomial weights re-encoded per call: N=2^15, 6 limbs, 2^30, 64 -> 64.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Config:
    key: str
    index: int          # seed index (1..5)
    log_n: int
    limbs: int
    log_scale: int
    d_in: int
    d_out: int
    weights: str        # "scalar" or "poly"
    encrypted: bool     # inputs are real encryptions (else uniform residues)
    description: str

    @property
    def n(self) -> int:
        return 1 << self.log_n

    @property
    def scale(self) -> float:
        return float(1 << self.log_scale)

    @property
    def macs(self) -> int:
        """Limb-coefficient modular MACs of one layer: d_out * d_in * 2 * L * N."""
        return self.d_out * self.d_in * 2 * self.limbs * self.n


CONFIGS = {
    "c1": Config("c1", 1, 10, 2, 25, 16, 16, "scalar", True,
                 "tiny ct x pt layer N=2^10 L=2 16->16 (encrypted, decrypt-checked)"),
    "c2": Config("c2", 2, 14, 4, 26, 768, 768, "scalar", False,
                 "GPT-2-124M attn-out projection N=2^14 L=4 768->768"),
    "c3": Config("c3", 3, 15, 6, 26, 768, 3072, "scalar", False,
                 "GPT-2-124M FFN up projection N=2^15 L=6 768->3072"),
    "c4": Config("c4", 4, 16, 8, 28, 1024, 6144, "scalar", False,
                 "Qwen3-0.6B gate+up projections N=2^16 L=8 1024->2x3072"),
    "c5": Config("c5", 5, 15, 6, 30, 64, 64, "poly", True,
                 "full-poly weights encoded per call N=2^15 L=6 64->64"),
}


def get(key: str) -> Config:
    return CONFIGS[key]
