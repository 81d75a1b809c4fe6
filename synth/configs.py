"""The five synthetic workloads, by shape.

c1  tiny fp32 dVLM step loop: 2 layers, d=256, 4 heads x 64, SwiGLU 1024,
    vocab 1024, one 12x12 crop (144 visual tokens), prompt 16, response 32,
    8 steps unmasking 4 per step, fixed view schedule 144,36,9,9,36,144,9,144.
c2  one 8B-shaped layer in bf16: d=4096, 32 heads x 128, SwiGLU 12288,
    vocab 126464; one 27x27 crop (729 tokens); prompt 32, response 128;
    64 steps unmasking 2 per step; high view for the first quarter of the
    steps, coarse view after.
c3  same layer, five 27x27 crops (3645 tokens), prompt 64, response 256,
    128 steps unmasking 2 per step; high view in the last eighth, coarse
    elsewhere.
c4  32-layer 8B-shaped stack, four crops (2916 tokens), prompt 48,
    response 128, 64 steps unmasking 2 per step; seeded i.i.d. level per step.
c5  ragged batch of 16 sequences through the 8B-shaped layer: 1-5 crops
    each, prompt 32-96, response 128, 64 steps unmasking 2 per step, the
    allocation policy choosing each sample's level per step.
"""

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    dtype: str            # "f32" or "bf16"
    n_layers: int
    d: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    grid: int             # crop side G (G x G tokens per crop)
    n_crops: int          # crops per sample (fixed-shape configs)
    prompt_len: int
    resp_len: int
    steps: int
    k: int                # tokens committed per step
    K: int = 3            # evidence levels
    n_seqs: int = 1
    schedule: str = "fixed"     # "fixed", "iid" or "policy"
    fixed_levels: Optional[Tuple[int, ...]] = None
    # ragged batch ranges (c5): crops U{lo..hi}, prompt U{lo..hi}
    crops_range: Optional[Tuple[int, int]] = None
    prompt_range: Optional[Tuple[int, int]] = None
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    weight_std: float = 0.02
    # allocation policy used when schedule == "policy" (LLaDA-V defaults)
    policy: dict = field(default_factory=lambda: dict(
        early=True, B=0.75, rho=0.20, alpha=1.0))

    @property
    def mask_id(self) -> int:
        return self.vocab - 1

    @property
    def n_visual(self) -> int:
        return self.n_crops * self.grid * self.grid


def _c2_levels():
    # high (level 2) for the first 25% of the 64 steps, coarse (level 0) after
    return tuple(2 if t < 16 else 0 for t in range(64))


def _c3_levels():
    # high for the last 1/8 of the 128 steps, coarse elsewhere
    return tuple(2 if t >= 112 else 0 for t in range(128))


CONFIGS = {
    1: Config(cid=1, name="tiny-f32", dtype="f32", n_layers=2, d=256,
              n_heads=4, head_dim=64, ffn=1024, vocab=1024, grid=12,
              n_crops=1, prompt_len=16, resp_len=32, steps=8, k=4,
              schedule="fixed", fixed_levels=(2, 1, 0, 0, 1, 2, 0, 2)),
    2: Config(cid=2, name="8b-layer-729", dtype="bf16", n_layers=1, d=4096,
              n_heads=32, head_dim=128, ffn=12288, vocab=126464, grid=27,
              n_crops=1, prompt_len=32, resp_len=128, steps=64, k=2,
              schedule="fixed", fixed_levels=_c2_levels()),
    3: Config(cid=3, name="8b-layer-3645", dtype="bf16", n_layers=1, d=4096,
              n_heads=32, head_dim=128, ffn=12288, vocab=126464, grid=27,
              n_crops=5, prompt_len=64, resp_len=256, steps=128, k=2,
              schedule="fixed", fixed_levels=_c3_levels()),
    4: Config(cid=4, name="8b-stack32-2916", dtype="bf16", n_layers=32,
              d=4096, n_heads=32, head_dim=128, ffn=12288, vocab=126464,
              grid=27, n_crops=4, prompt_len=48, resp_len=128, steps=64, k=2,
              schedule="iid"),
    5: Config(cid=5, name="8b-layer-ragged16", dtype="bf16", n_layers=1,
              d=4096, n_heads=32, head_dim=128, ffn=12288, vocab=126464,
              grid=27, n_crops=0, prompt_len=0, resp_len=128, steps=64, k=2,
              n_seqs=16, schedule="policy", crops_range=(1, 5),
              prompt_range=(32, 96)),
}


def get_config(cid: int) -> Config:
    return CONFIGS[int(cid)]


# Small shapes for parity tests: several tiles with ragged tails everywhere
# (pooling edges, GEMM rows, attention keys, vocabulary slabs).
TEST_CONFIGS = {
    11: Config(cid=11, name="mini-bf16", dtype="bf16", n_layers=2, d=256,
               n_heads=2, head_dim=128, ffn=512, vocab=1000, grid=7,
               n_crops=2, prompt_len=13, resp_len=37, steps=6, k=7,
               schedule="fixed", fixed_levels=(2, 0, 1, 1, 0, 2)),
    12: Config(cid=12, name="mini-bf16-ragged", dtype="bf16", n_layers=1,
               d=256, n_heads=2, head_dim=128, ffn=512, vocab=1000, grid=9,
               n_crops=0, prompt_len=0, resp_len=24, steps=4, k=6,
               n_seqs=5, schedule="policy", crops_range=(1, 3),
               prompt_range=(3, 40)),
    13: Config(cid=13, name="mini-f32-ragged", dtype="f32", n_layers=2,
               d=128, n_heads=2, head_dim=64, ffn=256, vocab=300, grid=5,
               n_crops=0, prompt_len=0, resp_len=20, steps=5, k=4,
               n_seqs=3, schedule="policy", crops_range=(1, 2),
               prompt_range=(2, 9)),
}


def get_any_config(cid: int) -> Config:
    return CONFIGS[int(cid)] if int(cid) in CONFIGS else TEST_CONFIGS[int(cid)]
