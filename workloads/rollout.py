"""Seeded rollout rounds for the scheduling simulation: R prompt groups of K samples.

``prompt_lens[g]`` (int32, R) is drawn uniform in ``[prompt_min, prompt_max]``.
Response lengths are log-normal with a per-group scale, since the K samples
of one prompt answer the same problem: group ``g`` draws
``m_g = median * exp(group_sigma * N(0, 1))`` and its samples
``resp_lens[g K + i] = round(m_g * exp(sample_sigma * N(0, 1)))``, clipped to
``[1, cap]``. The defaults give about 3.3k-token responses on average, the
paper's reported range (Section 5.3), with a marginal log-spread of
sqrt(0.5^2 + 0.3^2) = 0.58. Draw order from ``default_rng(seed)``: prompt
lengths, group scales, sample spreads. Nothing here schedules anything.
"""
from __future__ import annotations

import numpy as np


def make_rollout_workload(*, num_groups: int, group_size: int, seed: int, prompt_min: int = 128,
                          prompt_max: int = 1024, resp_median: float = 3000.0, group_sigma: float = 0.5,
                          sample_sigma: float = 0.3, resp_cap: int = 8192):
    rng = np.random.default_rng(seed)
    prompt = rng.integers(prompt_min, prompt_max + 1, num_groups).astype(np.int32)
    scale = np.log(resp_median) + group_sigma * rng.standard_normal(num_groups)
    z = np.repeat(scale, group_size) + sample_sigma * rng.standard_normal(num_groups * group_size)
    resp = np.clip(np.rint(np.exp(z)), 1, resp_cap).astype(np.int32)
    return prompt, resp
