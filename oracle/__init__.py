"""CPU oracle for the Hier-AVG round (Zhou & Cong, arXiv 1903.05133).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_1903_05133_amd``) never imports it, and this package imports nothing
from the product path: the two share no code, headers, constants or helpers.

What it is: a plain, slow, obviously correct numpy implementation of
Algorithm 1 (Sec. 3.1) in float64, written from the paper's statement of the
algorithm, plus its own implementation of the counter-based generator that
draws minibatches and synthesises the data (SplitMix64, Steele, Lea & Flood,
OOPSLA 2014).

Pins (what ties it to something other than itself) live in
``tests/test_oracle_*.py``: the SplitMix64 published output sequence, the
special cases Sec. 3.1 names (synchronous SGD, K-AVG), a plain minibatch-SGD
and momentum-SGD run through ``torch.autograd``/``torch.optim`` on the CPU in
float64, finite differences, the worker-average dynamics of the proof of
Thm 3.1, and the pure-noise variance that follows from the decomposition in
Lemma 1.  Every function here is pinned by one or more of these.  The paper
prints no parameter values after a round of the named workloads, so those
absolute values are checked only through the pinned functions that compute
them.

Modules:
  rng      -- SplitMix64 hash, the minibatch index draw, the exact normal
              surrogate, the synthetic data and initial-parameter recipes.
  method   -- per-model losses and gradients, the SGD / momentum update,
              group and global averaging, and one Hier-AVG round.
"""

from . import rng, method  # noqa: F401
