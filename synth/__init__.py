"""Seeded synthetic inputs for the compressed se_a descriptor.

This package only *prepares inputs*: atomic structures, neighbour lists, the
environment matrix R~ (weighting function s(r) and its normalisation, paper
Sec. II, Eq. (1) and the normalisation equations after it), random embedding
net weights, tabulation ranges and random upstream gradients dE/dT.

It contains none of the tabulation or descriptor arithmetic that the library
and the oracle implement (table construction, interval lookup, polynomial
evaluation, the contraction T = G^T R~, D = T T<^T and the backward pass).
Both the oracle (``oracle/``) and the GPU library read what this package
produces; neither is imported here.
"""
from .configs import CONFIGS, Config, get_config  # noqa: F401
from .system import Inputs, make_inputs  # noqa: F401
