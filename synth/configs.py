"""The five synthetic workloads (and small test variants).

Each stands in for one of the paper's systems (Sec. III: Cu, H2O, Al-Cu-Mg),
whose trained models and data sets are not available: structures are built
from a lattice of sites, neighbours are found within r_c, and the embedding
nets are random-initialised with the paper's layer sizes (Sec. III gives
(25, 50, 100) for Al-Cu-Mg; the same 1->25->50->100 shape is used for every
workload here, M' = 16).
"""
from dataclasses import dataclass, field, replace
from typing import Tuple

# Physical constants for the water box (density 1.0 g/cm^3).
_AVOGADRO = 6.02214076e23
_M_H2O = 18.015  # g/mol


@dataclass(frozen=True)
class Config:
    name: str
    kind: str                      # "fcc" or "water"
    ncell: int                     # cells per box edge (fcc cubic cells / water molecules)
    rc: float                      # cutoff r_c (Angstrom)
    rcs: float                     # smooth cutoff r_cs (Angstrom)
    sel: Tuple[int, ...]           # sel_alpha per neighbour type
    a: float = 3.634               # fcc lattice constant (Angstrom)
    jitter: float = 0.0            # Gaussian displacement sigma per component (Angstrom)
    type_probs: Tuple[float, ...] = (1.0,)  # fcc species probabilities
    density: float = 1.0           # water density (g/cm^3)
    widths: Tuple[int, ...] = (1, 25, 50, 100)  # embedding net layer widths
    m2: int = 16                   # M' (rows of S used for D)
    d1: float = 0.01               # table stride on the observed range
    d2: float = 0.1                # table stride on the extrapolation band
    dtype: str = "f64"             # "f64" or "f32"
    seed: int = 0                  # index spawned into the seed sequence

    @property
    def ntypes(self) -> int:
        return len(self.sel)

    @property
    def nnei(self) -> int:
        return int(sum(self.sel))

    @property
    def m1(self) -> int:
        return int(self.widths[-1])

    @property
    def natoms(self) -> int:
        n = self.ncell ** 3
        return 4 * n if self.kind == "fcc" else 3 * n

    @property
    def cell_edge(self) -> float:
        if self.kind == "fcc":
            return self.a
        vol_mol_cm3 = _M_H2O / _AVOGADRO / self.density
        return (vol_mol_cm3 * 1e24) ** (1.0 / 3.0)

    @property
    def box(self) -> float:
        return self.ncell * self.cell_edge

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS = (
    # 0: Cu-like, 256 atoms
    Config("cu256", "fcc", 4, rc=6.0, rcs=0.5, sel=(128,), a=3.634, jitter=0.1, seed=0),
    # 1: water-like, 4,096 molecules
    Config("water4096", "water", 16, rc=6.0, rcs=0.5, sel=(46, 92), seed=1),
    # 2: Al-Cu-Mg-like, 32,000 atoms
    Config("alcumg32000", "fcc", 20, rc=8.0, rcs=2.0, sel=(300, 60, 60), a=4.05,
           jitter=0.1, type_probs=(0.90, 0.05, 0.05), seed=2),
    # 3: Cu-like large, 1,048,576 atoms
    Config("cu1m", "fcc", 64, rc=8.0, rcs=2.0, sel=(512,), a=3.634, jitter=0.1, seed=3),
    # 4: water-like large, 110,592 molecules, fp32 storage
    Config("water110592", "water", 48, rc=6.0, rcs=0.5, sel=(46, 92), dtype="f32", seed=4),
)

# Small variants for CPU tests (box > 2 * (r_c + 2 * max displacement)).
TEST_CONFIGS = {
    "tiny_fcc": Config("tiny_fcc", "fcc", 3, rc=4.5, rcs=0.5, sel=(64,), a=3.634,
                       jitter=0.1, widths=(1, 4, 8, 16), m2=4, seed=10),
    "tiny_alloy": Config("tiny_alloy", "fcc", 3, rc=4.5, rcs=1.0, sel=(40, 20, 20), a=3.9,
                         jitter=0.1, type_probs=(0.6, 0.2, 0.2), widths=(1, 4, 8, 16),
                         m2=4, seed=11),
    "tiny_water": Config("tiny_water", "water", 5, rc=5.0, rcs=0.5, sel=(24, 48),
                         widths=(1, 4, 8, 16), m2=4, seed=12),
}


def get_config(key) -> Config:
    """Config by index (0..4), name, or test-variant name."""
    if isinstance(key, int):
        return CONFIGS[key]
    for c in CONFIGS:
        if c.name == key:
            return c
    if key in TEST_CONFIGS:
        return TEST_CONFIGS[key]
    raise KeyError(key)
