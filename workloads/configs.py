"""The five synthetic workloads: shapes, lengths, budgets and prune cadence.

Model shapes are those of the paper's evaluated models (Experimental Setup):
DeepSeek-R1-Distill-Llama-8B (32 layers, 32 query / 8 KV heads, head_dim 128)
and DeepSeek-R1-Distill-Qwen-7B (28 layers, 28 query / 4 KV heads).  The
datasets the paper decodes (Math500, an MMLU subset) are replaced by seeded
random keys/values whose per-layer attention concentration follows a Zipf
key-bias profile (see ``synth.py``).
"""
from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                 # "f32" or "bf16": storage type of q, K, V
    batch: int
    prompt: int                # cached rows per segment at the start (uniform configs)
    decode_steps: int          # generated tokens in the full run
    budget_frac: float         # global budget = floor(frac * T_b) * L per sequence
    prune_every: int           # decode steps between prune rounds
    recent: int
    sink: int = 0
    gamma: float = 0.99
    length_dist: str = "fixed"     # fixed | uniform | loguniform
    length_range: Tuple[int, int] = (0, 0)
    zipf: str = "iid"              # iid | ucurve | drift | fixed_weights | heavy_hitters
    zipf_range: Tuple[float, float] = (0.8, 1.6)
    epoch: int = 0                 # steps between re-drawn key directions (drift)
    notes: str = field(default="", compare=False)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


CONFIGS = {
    1: WorkloadConfig(
        name="tiny-fp32", num_layers=1, num_q_heads=4, num_kv_heads=2, head_dim=64, dtype="f32",
        batch=1, prompt=512, decode_steps=16, budget_frac=0.0, prune_every=16, recent=32,
        zipf="heavy_hitters",
        notes="1 layer, batch 1, 4/2 heads, D=64, fp32; 512 cached + 16 steps; one prune to 256, recent 32"),
    2: WorkloadConfig(
        name="llama8b-b8-2k+8k", num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
        batch=8, prompt=2048, decode_steps=8192, budget_frac=0.40, prune_every=512, recent=128,
        zipf="iid", zipf_range=(0.8, 1.6),
        notes="Llama-3-8B shapes, batch 8, 2k prompt + 8k generated, 40% budget, prune every 512, recent 128"),
    3: WorkloadConfig(
        name="qwen7b-b16-16k", num_layers=28, num_q_heads=28, num_kv_heads=4, head_dim=128, dtype="bf16",
        batch=16, prompt=16384, decode_steps=2048, budget_frac=0.30, prune_every=256, recent=256,
        zipf="ucurve",
        notes="Qwen-7B shapes (G=7), batch 16, 16k cached, 30% budget, prune every 256, recent 256"),
    4: WorkloadConfig(
        name="llama8b-b64-U8k32k", num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
        batch=64, prompt=0, decode_steps=4096, budget_frac=0.25, prune_every=256, recent=128,
        length_dist="uniform", length_range=(8192, 32768), zipf="drift", epoch=1000,
        notes="Llama-3-8B shapes, batch 64, lengths U[8k,32k], 25% budget, prune every 256, drift every 1k"),
    5: WorkloadConfig(
        name="llama8b-b128-logU1k64k", num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128,
        dtype="bf16", batch=128, prompt=0, decode_steps=1024, budget_frac=0.10, prune_every=128, recent=64,
        length_dist="loguniform", length_range=(1024, 65536), zipf="fixed_weights",
        notes="Llama-3-8B shapes, batch 128, lengths logU[1k,64k], 10% budget, prune every 128, recent 64"),
}

# Config 1 prunes once, to an absolute budget of 256 rows per segment.
TINY_BUDGET = 256
