"""Workload definitions: the shapes and parameter sets the detector is run on.

Pure data (no step of the method lives here).  Shapes stand in for the
paper's pipelines: k stages (shards) S, n canaries C, T tokens and hidden
size d = H (Section 3.1), with one malicious stage at the middle of the
pipeline as in the main factorial (Section 4.4).  All inputs are synthetic
and seeded; no dataset item or model weight is used.

Workloads
  tiny        4 x 8 x 16 x 256, stage 2 malicious, no outlier channels
  llama7b     8 x 64 x 128 x 4096 (32 layers as 8 shards), 41 outlier channels
  llama70b    16 x 256 x 256 x 8192 (80 layers as 16 shards), 82 outliers
  sweep       216-run factorial {8,16,32} shards x H {2048,4096,8192} x
              benign sigma {1e-4,1e-3} x tamper sigma {0.005,0.02,0.1} x
              {additive, sign flip, rescale, mixed}; 32 canaries x 64 tokens
  snr         16 x 128 x 128 x 4096, benign sigma at 20 log-spaced values in
              [1e-4, 1e-1], Gaussian and Student-t noise, tamper 0.02
  paper       12 x 100 x 48 x 768 (the paper's GPT-2 / Pythia-160M shape),
              block-scaled benign noise sigma_hw = 0.002, the six attacks
  substudies  the depth, position, collusion, frontier and SNR substudies
              on the paper's shape with the live error carried between stages
"""
from dataclasses import dataclass, field
from typing import List, Tuple

NOISE_ELEMENTWISE = 0
NOISE_BLOCK = 1
DIST_GAUSS = 0
DIST_T3 = 1
T_ADD = 1
T_FLIP = 2
T_SCALE = 4
T_MIXED = T_ADD | T_FLIP | T_SCALE
BASE_BENIGN = 0
BASE_CLEAN = 1

SEED = 0
OUTLIER_GAIN = 20.0


@dataclass(frozen=True)
class Run:
    """One simulated live pass over a reference set plus its scoring."""
    cfg_id: int
    benign_mode: int = NOISE_ELEMENTWISE
    benign_dist: int = DIST_GAUSS
    sigma_b: float = 1e-3
    tamper: int = T_ADD
    eps: float = 0.0        # Gaussian tamper magnitude (times the block rms)
    flip_p: float = 0.0     # sign-flip fraction (1.0 = the paper's full flip)
    scale: float = 1.0      # rescale factor 1 + alpha
    tamper_base: int = BASE_BENIGN
    exact_norm: bool = False  # Gaussian tamper scaled to exactly eps ||v|| (Section 3.2)
    carry: float = 0.0        # propagation gain of the live error between stages
    label: str = ""


@dataclass(frozen=True)
class RefSet:
    """One reference set [S][C][T][H] and the runs made against it."""
    ref_set_id: int
    S: int
    C: int
    T: int
    H: int
    n_out: int
    mal_shards: Tuple[int, ...]
    runs: Tuple[Run, ...] = field(default_factory=tuple)

    @property
    def mal_mask(self) -> int:
        m = 0
        for s in self.mal_shards:
            m |= 1 << s
        return m

    @property
    def elems(self) -> int:
        return self.S * self.C * self.T * self.H

    @property
    def block_elems(self) -> int:
        return self.T * self.H


@dataclass(frozen=True)
class Workload:
    name: str
    ref_sets: Tuple[RefSet, ...]
    seed: int = SEED

    @property
    def n_runs(self) -> int:
        return sum(len(r.runs) for r in self.ref_sets)


def n_outliers(H: int, frac: float = 0.01) -> int:
    """Number of outlier channels: the nearest integer to frac * H."""
    return int(frac * H + 0.5)


def tiny() -> Workload:
    rs = RefSet(0, 4, 8, 16, 256, 0, (2,),
                (Run(0, sigma_b=1e-3, tamper=T_ADD, eps=0.05, label="add0.05"),))
    return Workload("tiny", (rs,))


def llama7b() -> Workload:
    S, H = 8, 4096
    runs = (Run(0, sigma_b=1e-3, tamper=T_ADD, eps=0.01, label="add0.01"),
            Run(1, sigma_b=1e-3, tamper=T_ADD, eps=0.05, label="add0.05"))
    return Workload("llama7b", (RefSet(0, S, 64, 128, H, n_outliers(H), (S // 2,), runs),))


def llama70b() -> Workload:
    S, H = 16, 8192
    runs = (Run(0, sigma_b=1e-3, tamper=T_ADD, eps=0.05, label="add0.05"),
            Run(1, sigma_b=1e-3, tamper=T_FLIP, flip_p=0.001, label="flip0.001"),
            Run(2, sigma_b=1e-3, tamper=T_SCALE, scale=1.05, label="scale1.05"))
    return Workload("llama70b", (RefSet(0, S, 256, 256, H, n_outliers(H), (S // 2,), runs),))


SWEEP_SHARDS = (8, 16, 32)
SWEEP_HIDDEN = (2048, 4096, 8192)
SWEEP_SIGMA_B = (1e-4, 1e-3)
SWEEP_SIGMA_T = (0.005, 0.02, 0.1)
SWEEP_TYPES = (("add", T_ADD), ("flip", T_FLIP), ("scale", T_SCALE), ("mixed", T_MIXED))


def _typed_run(cfg_id, sigma_b, sigma_t, tname, tflags):
    return Run(cfg_id, sigma_b=sigma_b, tamper=tflags,
               eps=sigma_t if tflags & T_ADD else 0.0,
               flip_p=sigma_t if tflags & T_FLIP else 0.0,
               scale=1.0 + sigma_t if tflags & T_SCALE else 1.0,
               label=f"{tname}:sb{sigma_b:g}:st{sigma_t:g}")


def sweep() -> Workload:
    """The 216-run factorial; cfg_id follows the nested order
    (shards, hidden, benign sigma, tamper sigma, tamper type)."""
    sets = []
    cfg_id = 0
    for S in SWEEP_SHARDS:
        for H in SWEEP_HIDDEN:
            runs = []
            for sb in SWEEP_SIGMA_B:
                for st in SWEEP_SIGMA_T:
                    for tname, tflags in SWEEP_TYPES:
                        runs.append(_typed_run(cfg_id, sb, st, tname, tflags))
                        cfg_id += 1
            sets.append(RefSet(len(sets), S, 32, 64, H, n_outliers(H), (S // 2,), tuple(runs)))
    return Workload("sweep", tuple(sets))


def snr_sigmas() -> List[float]:
    """20 benign noise levels, log-spaced from 1e-4 to 1e-1."""
    return [10.0 ** (-4.0 + 3.0 * j / 19.0) for j in range(20)]


def snr() -> Workload:
    S, H = 16, 4096
    runs = []
    for j, sb in enumerate(snr_sigmas()):
        for dist, dname in ((DIST_GAUSS, "gauss"), (DIST_T3, "t3")):
            runs.append(Run(len(runs), benign_dist=dist, sigma_b=sb, tamper=T_ADD, eps=0.02,
                            label=f"{dname}:sb{sb:.3g}"))
    return Workload("snr", (RefSet(0, S, 128, 128, H, n_outliers(H), (S // 2,), tuple(runs)),))


def paper() -> Workload:
    """The paper's own pipeline shape: 12 stages, 100 canaries of 48 tokens,
    d = 768, malicious stage floor(k/2) = 6 counted from 1 (index 5 here),
    block-scaled benign noise at sigma_hw = 0.002 and the six attacks, the
    Gaussian ones with the exact norm eps ||v||."""
    S, H = 12, 768
    runs = []
    for eps in (0.02, 0.05, 0.10, 0.20):
        runs.append(Run(len(runs), benign_mode=NOISE_BLOCK, sigma_b=0.002, tamper=T_ADD,
                        eps=eps, exact_norm=True, label=f"gauss{eps:g}"))
    runs.append(Run(len(runs), benign_mode=NOISE_BLOCK, sigma_b=0.002, tamper=T_FLIP,
                    flip_p=1.0, label="signflip"))
    runs.append(Run(len(runs), benign_mode=NOISE_BLOCK, sigma_b=0.002, tamper=T_SCALE,
                    scale=1.10, label="rescale0.10"))
    return Workload("paper", (RefSet(0, S, 100, 48, H, n_outliers(H), (S // 2 - 1,),
                                     tuple(runs)),))


SUBSTUDY_CARRY = 0.7
SUBSTUDY_DEPTHS = (2, 4, 6, 8, 10, 12)
SUBSTUDY_POSITIONS = (0, 2, 5, 8, 11)          # first ... last of 12 stages
SUBSTUDY_COLLUDERS = (1, 2, 3, 4)
SUBSTUDY_EPS = (0.10, 0.05, 0.02, 0.01, 0.005, 0.002, 0.001)
SUBSTUDY_SIGMA_HW = (0.002, 0.01, 0.02, 0.05, 0.1, 0.2)


def colluder_positions(k: int, c: int) -> Tuple[int, ...]:
    """c colluders spaced uniformly over k stages (0-indexed): the j-th at
    floor(k (j + 1) / (c + 1)) - 1, so c = 1 is the middle stage floor(k/2)."""
    return tuple(k * (j + 1) // (c + 1) - 1 for j in range(c))


def substudies() -> Workload:
    """Sections 4.4 and 5.3-5.5 on the paper's shape (100 canaries x 48 tokens
    x d = 768, block noise sigma_hw = 0.002), with the live error of each
    stage carried into the next (gain SUBSTUDY_CARRY):
      depth      k in {2, ..., 12}, attacker at the middle, Gaussian 0.05
      position   k = 12, attacker at 5 positions from first to last
      collusion  k = 12, 1..4 colluders spaced uniformly
      frontier   k = 12, Gaussian eps from 0.10 down to 0.001
      snr        k = 12, Gaussian 0.05, sigma_hw raised from 0.002 to 0.2
                 (Section 5.4)
    Every Gaussian attack is the paper's exact-norm one, eps ||v|| with v the
    attacker's untampered live output given the error carried in from
    upstream (Section 3.2).
    Each configuration is one reference set with one run; configurations of
    one shape share their references (same ref_set_id)."""
    C, T, H = 100, 48, 768
    n_out = n_outliers(H)
    sets = []

    def add(name, S, mal, eps, sigma_hw=0.002):
        run = Run(len(sets), benign_mode=NOISE_BLOCK, sigma_b=sigma_hw, tamper=T_ADD, eps=eps,
                  exact_norm=True, carry=SUBSTUDY_CARRY, label=name)
        sets.append(RefSet(S, S, C, T, H, n_out, tuple(mal), (run,)))

    for k in SUBSTUDY_DEPTHS:
        add(f"depth:k{k}", k, (k // 2 - 1,), 0.05)
    for pos in SUBSTUDY_POSITIONS:
        add(f"position:{pos}", 12, (pos,), 0.05)
    for c in SUBSTUDY_COLLUDERS:
        add(f"collusion:c{c}", 12, colluder_positions(12, c), 0.05)
    for eps in SUBSTUDY_EPS:
        add(f"frontier:eps{eps:g}", 12, (5,), eps)
    for sigma in SUBSTUDY_SIGMA_HW:
        add(f"snr:sigma{sigma:g}", 12, (5,), 0.05, sigma)
    return Workload("substudies", tuple(sets))


WORKLOADS = {"tiny": tiny, "llama7b": llama7b, "llama70b": llama70b, "sweep": sweep,
             "snr": snr, "paper": paper, "substudies": substudies}


def get(name: str) -> Workload:
    return WORKLOADS[name]()
