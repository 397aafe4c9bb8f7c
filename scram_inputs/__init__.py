"""Seeded synthetic inputs for the SCRAM hot path.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no part of the method's arithmetic (no scores, no PatchMatch, no
softmax): it only draws Q, K, V images with the two properties the method
relies on (Section 4.1): spatial coherence -- queries near each other match
keys shifted by the same amount -- and sparse structure -- each query's best
keys sit in one small blob.

Recipe (all numpy, fp32, deterministic from ``data_seed``):

1. K: i.i.d. N(0, 1) of shape [S, Hk, Wk, d], Gaussian-blurred per channel
   along both grid axes (sigma px, truncated at 4 sigma, reflecting border),
   then normalised to unit L2 norm per pixel.
2. A displacement field f: U(-1, 1) of shape [S, Hq, Wq, 2], blurred with
   2 sigma, rescaled so that max_p |f(p)|_2 = F.
3. Target key pixel tau(p) = clamp(round(s * p + f(p))) into the key grid;
   a Bernoulli(outlier_frac) subset of queries gets a uniform random target.
4. Q(p) = 4 * K(tau(p)) + 0.1 * N(0, 1) per element.
5. V: i.i.d. N(0, 1) of shape [S, Hk, Wk, dv].
6. bf16 workloads round these fp32 arrays to bf16 (nearest-even); every
   consumer reads the same rounded values.
"""
from __future__ import annotations

from .configs import CONFIGS, EXTRA, HEADLINE, Workload, get  # noqa: F401
from .synth import make, make_arrays  # noqa: F401
