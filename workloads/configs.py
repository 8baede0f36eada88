"""The five decode-attention workloads, with their size and distribution recipes.

Group structure follows the GRPO rollout the paper describes: every prompt is
sampled K times (K = G here), and the K responses share one prompt prefix
(Section 2.1; Section 5.1 uses K = 8). Head counts and head_dim are the
Qwen3-1.7B attention layer (Hq = 16, Hkv = 8, d = 128; Section 5.1 names the
model). Length distributions stand in for the reasoning workloads of
Section 5.1, whose responses average 3.3k-3.6k tokens (Section 5.3); the
datasets themselves are not used.
"""
from dataclasses import dataclass
from typing import Optional


@dataclass(frozen=True)
class DecodeConfig:
    cid: int
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    groups: int                  # prompt groups present in the batch
    group_size: int              # G responses sampled per prompt
    prefix: tuple                # ("fixed", P) or ("uniform", lo, hi)
    resp: tuple                  # ("uniform", lo, hi) or ("lognormal", median, sigma, cap)
    live: Optional[tuple] = None  # ("uniform", lo, hi, total) partially finished groups
    random_group_map: bool = False
    k_mult: float = 1.0          # K drawn as k_mult * N(0, 1)
    append: bool = False         # one new token per sequence appended before attention
    kv_dtype: str = "bf16"       # "bf16" or "fp8"
    page_size: int = 16

    @property
    def seed(self) -> int:
        return 1000 + self.cid

    @property
    def max_prefix(self) -> int:
        return self.prefix[1] if self.prefix[0] == "fixed" else self.prefix[2]

    @property
    def max_resp(self) -> int:
        """Largest number of response tokens in the cache at attention time."""
        r = self.resp
        cap = r[2] if r[0] == "uniform" else r[3]
        return cap + (1 if self.append else 0)


CONFIGS = {
    1: DecodeConfig(1, "tiny: 1 group x G=4, Hq=4 Hkv=2 d=64, prefix 128, resp U[32,64]",
                    num_q_heads=4, num_kv_heads=2, head_dim=64, groups=1, group_size=4,
                    prefix=("fixed", 128), resp=("uniform", 32, 64)),
    2: DecodeConfig(2, "qwen3-1.7b layer: 32 prompts x G=8, prefix U[64,512], resp U[0,4096], K*0.5",
                    num_q_heads=16, num_kv_heads=8, head_dim=128, groups=32, group_size=8,
                    prefix=("uniform", 64, 512), resp=("uniform", 0, 4096), k_mult=0.5),
    3: DecodeConfig(3, "reasoning tail: 64 prompts x G=16, prefix 256, resp lognormal(1500, 0.9) cap 8192, +append",
                    num_q_heads=16, num_kv_heads=8, head_dim=128, groups=64, group_size=16,
                    prefix=("fixed", 256), resp=("lognormal", 1500.0, 0.9, 8192), append=True),
    4: DecodeConfig(4, "frontier-mixed: 512 live of 128 groups x G=8, prefix U[128,1024], resp U[0,16384], random map",
                    num_q_heads=16, num_kv_heads=8, head_dim=128, groups=128, group_size=8,
                    prefix=("uniform", 128, 1024), resp=("uniform", 0, 16384),
                    live=("uniform", 1, 8, 512), random_group_map=True),
    5: DecodeConfig(5, "fp8 long context: 16 prompts x G=16, prefix 256, resp U[8192,32768], +append, e4m3 KV",
                    num_q_heads=16, num_kv_heads=8, head_dim=128, groups=16, group_size=16,
                    prefix=("fixed", 256), resp=("uniform", 8192, 32768), append=True, kv_dtype="fp8"),
}


def config_by_id(cid: int) -> DecodeConfig:
    return CONFIGS[int(cid)]
