"""Named synthetic workloads shaped like the paper's video-DiT attention calls.

Token counts follow Sec. 5.1: Wan2.1 at 480p is 21 latent frames of 30 x 52
tokens (32 760), Wan2.1-14B at 720p is 21 frames of 45 x 80 (75 600).  The
sequence is padded to a multiple of the block size with ordinary N(0,1)
tokens so that every block is full and FLOP counts are exact; the ragged
lengths are separate correctness cases.  Head counts and head dimension
(12 heads for the 1.3B model, 40 for the 14B model, d = 128) are the Wan2.1
architectures'; the block size is the paper's B = 128 (Sec. 4.1.1, Sec. 4.3.2).
"""

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int                      # sequence length handed to the kernel
    d: int
    blk_q: int
    blk_k: int
    grid: Tuple[int, int, int]  # (frames, rows, cols) of the latent token grid
    mask_kind: str              # "structured" | "uniform" | "dense"
    rho: Optional[float] = None
    rho_range: Optional[Tuple[float, float]] = None
    head_scale_range: Optional[Tuple[float, float]] = None
    w_t: Optional[int] = None
    n_globals: Optional[int] = None
    mask_seed: int = 1000
    data_seed: int = 2000
    sample_seed: int = 3000
    extra: dict = field(default_factory=dict)

    @property
    def n_qb(self):
        return -(-self.N // self.blk_q)

    @property
    def n_kb(self):
        return -(-self.N // self.blk_k)

    @property
    def scale(self):
        return 1.0 / float(self.d) ** 0.5

    def with_(self, **kw):
        return replace(self, **kw)


def _pad(n, blk):
    return -(-n // blk) * blk


TINY = Workload(
    name="tiny_h1_n1024_d64_blk64", B=1, H=1, N=1024, d=64, blk_q=64, blk_k=64,
    grid=(4, 16, 16), mask_kind="structured", rho=0.25, w_t=1, n_globals=0,
    mask_seed=1000, data_seed=2000, sample_seed=3000)

WAN13B_480P = Workload(
    name="wan2.1-1.3b_480p_h12_n32768_d128_blk128", B=1, H=12, N=_pad(21 * 30 * 52, 128),
    d=128, blk_q=128, blk_k=128, grid=(21, 30, 52), mask_kind="structured",
    rho_range=(0.15, 0.5), head_scale_range=(0.5, 2.0),
    mask_seed=1001, data_seed=2001, sample_seed=3001)

WAN14B_480P = Workload(
    name="wan2.1-14b_480p_h40_n32768_d128_blk128", B=1, H=40, N=_pad(21 * 30 * 52, 128),
    d=128, blk_q=128, blk_k=128, grid=(21, 30, 52), mask_kind="structured",
    rho_range=(0.05, 0.6), head_scale_range=(0.5, 2.0),
    mask_seed=1002, data_seed=2002, sample_seed=3002)

WAN14B_720P = Workload(
    name="wan2.1-14b_720p_h40_n75648_d128_blk128", B=1, H=40, N=_pad(21 * 45 * 80, 128),
    d=128, blk_q=128, blk_k=128, grid=(21, 45, 80), mask_kind="structured",
    rho_range=(0.05, 0.3), head_scale_range=(0.5, 2.0),
    mask_seed=1003, data_seed=2003, sample_seed=3003)


def sweep_point(rho, blk, kind):
    """Density / block-size sweep point: H=40, N=32768, d=128, s_h = 1."""
    tag = "dense" if rho >= 1.0 else kind
    return Workload(
        name="sweep_h40_n32768_d128_blk%d_%s_rho%.2f" % (blk, tag, rho),
        B=1, H=40, N=32768, d=128, blk_q=blk, blk_k=blk, grid=(21, 30, 52),
        mask_kind="dense" if rho >= 1.0 else kind, rho=None if rho >= 1.0 else rho,
        mask_seed=1004, data_seed=2004, sample_seed=3004)


SWEEP_RHOS = (1.0, 0.5, 0.25, 0.1, 0.05)
SWEEP_BLKS = (64, 128)
SWEEP_KINDS = ("structured", "uniform")

NAMED = {w.name: w for w in (TINY, WAN13B_480P, WAN14B_480P, WAN14B_720P)}
SHORT = {"tiny": TINY, "1.3b-480p": WAN13B_480P, "14b-480p": WAN14B_480P,
         "14b-720p": WAN14B_720P}
