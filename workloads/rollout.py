"""Seeded rollout rounds for the scheduling simulation: R prompt groups of K samples.

``prompt_lens[g]`` (int32, R) is drawn uniform in ``[prompt_min, prompt_max]``;
``resp_lens[g K + i]`` (int32, R K) is ``round(exp(N(ln median, sigma^2)))``
clipped to ``[1, cap]``, so responses average about 3.5k tokens with the
defaults, the paper's reported range (Section 5.3). Draw order from
``default_rng(seed)``: prompt lengths, then response lengths. Nothing here
schedules anything.
"""
from __future__ import annotations

import numpy as np


def make_rollout_workload(*, num_groups: int, group_size: int, seed: int, prompt_min: int = 128,
                          prompt_max: int = 1024, resp_median: float = 3000.0, resp_sigma: float = 0.6,
                          resp_cap: int = 8192):
    rng = np.random.default_rng(seed)
    prompt = rng.integers(prompt_min, prompt_max + 1, num_groups).astype(np.int32)
    z = rng.standard_normal(num_groups * group_size)
    resp = np.clip(np.rint(np.exp(np.log(resp_median) + resp_sigma * z)), 1, resp_cap).astype(np.int32)
    return prompt, resp
