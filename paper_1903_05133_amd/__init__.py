"""Hier-AVG (Zhou & Cong, arXiv 1903.05133) hot path on one MI355X: P learners
as rows of one replica array, local SGD, cluster means and the global mean as
hand-written HIP kernels behind the C ABI of include/hieravg.h."""

from . import native  # noqa: F401
from .hieravg import HierAvg, config  # noqa: F401
