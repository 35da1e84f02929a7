"""The five synthetic workloads, named by what they are.

They stand in for the paper's LongBench traces on LWM-7B / Llama-3-8B-262k
(Section 5.1): model shapes are Llama-3-8B-like (32 query / 8 KV heads) and
a Qwen-like GQA-7 shape, head_dim 128, with a 2048- or 4096-token budget
(Section 5.2 uses 2048).  Values are synthetic: K, V ~ N(0,1) times a
per-channel scale U[0.5, 2]; q ~ N(0,1).
"""
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Config:
    name: str
    B: int                 # sequences in the batch
    Hq: int                # query heads
    Hkv: int               # KV heads
    d: int                 # head dim
    blk: int               # tokens per block
    k: int                 # blocks selected per (sequence, KV head)
    ctx: int = 0           # context tokens (fixed length)
    ctx_range: tuple = ()  # (lo, hi) for ragged lengths, rounded to blk
    n_plant: int = 0       # planted critical blocks per (sequence, KV head)
    plant_shift: float = 1.5
    placement: str = "hbm"  # "hbm": all KV resident in HBM; "host": pinned host pool + HBM cache
    cache_frac: float = 0.0  # HBM cache slots per unit as a fraction of its blocks
    steps: int = 1         # timed decode steps (after one warm-up step for "host")
    drift: float = 0.0     # query drift sigma per step
    layers: int = 1
    notes: str = field(default="", compare=False)

    @property
    def G(self):
        return self.Hq // self.Hkv

    @property
    def record_bytes(self):
        return 2 * self.blk * self.d * 2

    @property
    def nblk_max(self):
        if self.ctx_range:
            return self.ctx_range[1] // self.blk
        return self.ctx // self.blk


CONFIGS = [
    Config("tiny-b2-h8kv2-ctx4k-blk16-k16", B=2, Hq=8, Hkv=2, d=128, blk=16, k=16, ctx=4096,
           n_plant=8, placement="hbm", steps=1),
    Config("llama3-8b-b32-ctx32k-blk16-k128", B=32, Hq=32, Hkv=8, d=128, blk=16, k=128, ctx=32768,
           n_plant=64, placement="hbm", steps=1),
    Config("hier-b64-ctx128k-blk16-k128-cache25", B=64, Hq=32, Hkv=8, d=128, blk=16, k=128, ctx=131072,
           placement="host", cache_frac=0.25, steps=16, drift=0.3),
    Config("layers32-b16-ragged8k64k-blk16-k128-cache30", B=16, Hq=32, Hkv=8, d=128, blk=16, k=128,
           ctx_range=(8192, 65536), placement="host", cache_frac=0.30, steps=8, drift=0.3, layers=32),
    Config("qwen-gqa7-b48-ctx128k-blk8-k512-cache15", B=48, Hq=28, Hkv=4, d=128, blk=8, k=512, ctx=131072,
           placement="host", cache_frac=0.15, steps=8, drift=0.6),
]


def get(i_or_name):
    if isinstance(i_or_name, int):
        return CONFIGS[i_or_name]
    for c in CONFIGS:
        if c.name == i_or_name:
            return c
    raise KeyError(i_or_name)
