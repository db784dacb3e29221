"""The five synthetic workloads of the scheduler core, with their sizes.

Every length is an integer token count.  The length model is the heavy-tailed
lognormal family the paper's workloads motivate (Sec. 1 and App. A: skewed,
heavy-tailed output lengths); prompts of the two largest workloads mix in a
long-context share.  Values not fixed by the workload statement are marked
"reading".
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class LogNormal:
    """Lengths ``clip(rint(exp(mu + sigma * z)), lo, hi)``, z ~ N(0, 1)."""
    mu: float
    sigma: float
    lo: int
    hi: int


@dataclass(frozen=True)
class PromptMix:
    """With probability ``long_frac`` a prompt is uniform on [long_lo, long_hi],
    otherwise it follows ``base``."""
    base: LogNormal
    long_frac: float = 0.0
    long_lo: int = 0
    long_hi: int = 0


@dataclass(frozen=True)
class Workload:
    name: str
    decoders: int            # D, the decode instances (Sec. 3.3)
    residents: int           # requests resident on each decoder
    arrivals: int            # A, requests to place in one batch
    capacities: tuple        # C_k in tokens; each decoder draws one uniformly
    prompt: PromptMix        # L_prom
    output: LogNormal        # true L_out
    pred_sigma: float        # predictor = true * lognormal(0, pred_sigma)
    n_cal: int               # calibration residuals (Sec. 3.2)
    buckets: int             # length buckets of the per-bucket quantile
    alphas_ppm: tuple        # target miscoverage alpha, in parts per million
    queue_fixed: int | None  # pending requests per decoder if fixed, else None
    queue_max: int = 63      # otherwise Q_d ~ U{0..queue_max} (reading)
    seed: int = 0
    bytes_per_token: int | None = None   # KV bytes per token (App. A note)
    wait_mean_ms: float = 250.0          # queue wait ~ floor(Exp(mean)) (reading)
    max_wait_ms: int = 1000              # starvation threshold (Sec. 4)
    gen_frac: float = 1.0                # residents generated g = floor(f * gen_frac * true), f ~ U[0,1)
    notes: dict = field(default_factory=dict)

    @property
    def u_max(self) -> int:
        """Largest admissible upper bound: the output-length clip (reading)."""
        return self.output.hi

    @property
    def pairs(self) -> int:
        return self.decoders * self.arrivals


_SHORT_PROMPT = PromptMix(LogNormal(6.0, 1.0, 16, 4096))
_MID_PROMPT = PromptMix(LogNormal(7.0, 1.0, 16, 16384))
_LONG_MIX = PromptMix(LogNormal(7.0, 1.0, 16, 16384), 0.2, 32768, 131072)
_HETERO = (131072, 262144, 524288)

WORKLOADS = {
    "tiny": Workload(
        name="tiny", decoders=4, residents=64, arrivals=256, capacities=(65536,),
        prompt=_SHORT_PROMPT, output=LogNormal(6.0, 1.2, 1, 8192), pred_sigma=0.3,
        n_cal=1000, buckets=4, alphas_ppm=(100000,), queue_fixed=None, seed=0),
    "small": Workload(
        name="small", decoders=16, residents=256, arrivals=4096, capacities=(262144,),
        prompt=_SHORT_PROMPT, output=LogNormal(6.0, 1.2, 1, 8192), pred_sigma=0.3,
        n_cal=20000, buckets=16, alphas_ppm=(50000, 100000), queue_fixed=None, seed=1,
        bytes_per_token=131072),
    "medium": Workload(
        name="medium", decoders=64, residents=1024, arrivals=65536, capacities=(262144,),
        prompt=_MID_PROMPT, output=LogNormal(6.5, 1.5, 1, 32768), pred_sigma=0.5,
        n_cal=200000, buckets=32, alphas_ppm=(100000,), queue_fixed=None, seed=2),
    "large": Workload(
        name="large", decoders=256, residents=4096, arrivals=262144, capacities=_HETERO,
        prompt=_LONG_MIX, output=LogNormal(6.5, 1.5, 1, 32768), pred_sigma=0.5,
        n_cal=1000000, buckets=64, alphas_ppm=(50000,), queue_fixed=None, seed=3),
    "xlarge": Workload(
        name="xlarge", decoders=1024, residents=2048, arrivals=1048576, capacities=_HETERO,
        prompt=_LONG_MIX, output=LogNormal(7.0, 1.8, 1, 65536), pred_sigma=0.5,
        n_cal=4000000, buckets=128, alphas_ppm=(100000,), queue_fixed=512, seed=4),
}

# Not one of the five: the large shape with residents early in long outputs
# (short prompts, few tokens generated, outputs of thousands of tokens), so
# that every decoder's occupancy keeps growing long after its first events
# and placement needs the event records of the hot and full walks instead of
# the flat region that every decoder of `large` reaches at once.
WORKLOADS["large_growing"] = Workload(
    name="large_growing", decoders=256, residents=4096, arrivals=262144, capacities=_HETERO,
    prompt=PromptMix(LogNormal(4.0, 1.0, 1, 512)), output=LogNormal(8.5, 1.0, 1, 32768), pred_sigma=0.5,
    n_cal=1000000, buckets=64, alphas_ppm=(50000,), queue_fixed=None, seed=13, gen_frac=0.05)

# Workloads in size order; index i is the i-th workload of the scheduler-core
# benchmark statement (tiny .. xlarge).
ORDER = ("tiny", "small", "medium", "large", "xlarge")


def describe(w: Workload) -> str:
    return (f"{w.decoders} decoders x {w.residents} residents, {w.arrivals} arrivals, "
            f"{w.n_cal} calibration residuals in {w.buckets} buckets")
