"""The five synthetic workloads (shapes and draw parameters only).

They stand in for the replayed Claude Code / SWE-bench Pro traces of the
paper's evaluation (Sec. 6.1), which are not available: program sizes follow
long-context agent sessions, idleness windows follow the busy/idle two-phase
structure of Sec. 3.3, and the KV geometry is that of the named models.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class KVConfig:
    name: str
    layers: int
    planes: int          # 2 for separate K and V, 1 for a compressed latent
    block_tokens: int
    row_bytes: int       # bytes of one token in one (layer, plane)
    dtype: str           # 'fp16' | 'bf16' (element type of the synthetic KV values)
    programs: int
    ctx_kind: str        # 'uniform' | 'lognormal'
    ctx_median: int      # lognormal median (tokens); unused for 'uniform'
    ctx_lo: int
    ctx_hi: int
    busy_frac: float
    gpu_pct: float       # GPU budget, percent of total KV bytes
    frag: str            # 'shuffled' (uniform permutation) | 'chunked' (geometric chunks, mean 4 pages)
    seed: int
    min_blocks: int = 0  # pool size floor (the tiny pool has 256 blocks)
    steps: int = 0       # churn steps
    flip_frac: float = 0.0
    pct_swing: tuple = field(default=(0.0, 0.0))  # (centre, amplitude) of an oscillating GPU budget

    @property
    def run_bytes(self) -> int:
        """Bytes of one (layer, plane, page): block_tokens rows."""
        return self.block_tokens * self.row_bytes

    @property
    def block_bytes(self) -> int:
        """Bytes of one page over every layer and plane."""
        return self.layers * self.planes * self.run_bytes

    @property
    def bytes_per_token(self) -> int:
        return self.layers * self.planes * self.row_bytes


SIGMA_CTX = 0.5        # lognormal sigma of context lengths
WINDOW_K = 5           # cycles in the idleness window (the paper uses k = 5)
R_MEDIAN, R_SIGMA = 2.0, 0.5            # reasoning (inference) interval, seconds
A_BUSY_MEDIAN, A_IDLE_MEDIAN, A_SIGMA = 1.0, 60.0, 1.0   # tool-call interval, seconds
FRAG_MEAN_CHUNK = 4.0

TINY = KVConfig("tiny", layers=2, planes=2, block_tokens=16, row_bytes=4 * 64 * 2, dtype="fp16",
                programs=8, ctx_kind="uniform", ctx_median=0, ctx_lo=100, ctx_hi=2000, busy_frac=0.5,
                gpu_pct=60.0, frag="shuffled", seed=1, min_blocks=256)
LLAMA3_8B = KVConfig("llama3_8b", layers=32, planes=2, block_tokens=16, row_bytes=8 * 128 * 2, dtype="bf16",
                     programs=64, ctx_kind="lognormal", ctx_median=16384, ctx_lo=4096, ctx_hi=65536,
                     busy_frac=0.5, gpu_pct=50.0, frag="chunked", seed=2)
LLAMA3_70B = KVConfig("llama3_70b", layers=80, planes=2, block_tokens=16, row_bytes=8 * 128 * 2, dtype="bf16",
                      programs=64, ctx_kind="lognormal", ctx_median=6144, ctx_lo=2048, ctx_hi=24576,
                      busy_frac=0.3, gpu_pct=60.0, frag="chunked", seed=3)
# one rank's share of the Llama-3-70B programs under tensor parallelism of 2:
# the same programs (same seed), half of the 8 KV heads per rank, so 1 KiB rows
# and 16 KiB runs
LLAMA3_70B_TP2 = KVConfig("llama3_70b_tp2", layers=80, planes=2, block_tokens=16, row_bytes=4 * 128 * 2,
                          dtype="bf16", programs=64, ctx_kind="lognormal", ctx_median=6144, ctx_lo=2048,
                          ctx_hi=24576, busy_frac=0.3, gpu_pct=60.0, frag="chunked", seed=3)
# the same share at tensor parallelism 4 and 8: 2 and 1 KV heads per rank, 512-B and 256-B rows, 8 and 4 KiB runs
LLAMA3_70B_TP4 = KVConfig("llama3_70b_tp4", layers=80, planes=2, block_tokens=16, row_bytes=2 * 128 * 2,
                          dtype="bf16", programs=64, ctx_kind="lognormal", ctx_median=6144, ctx_lo=2048,
                          ctx_hi=24576, busy_frac=0.3, gpu_pct=60.0, frag="chunked", seed=3)
LLAMA3_70B_TP8 = KVConfig("llama3_70b_tp8", layers=80, planes=2, block_tokens=16, row_bytes=1 * 128 * 2,
                          dtype="bf16", programs=64, ctx_kind="lognormal", ctx_median=6144, ctx_lo=2048,
                          ctx_hi=24576, busy_frac=0.3, gpu_pct=60.0, frag="chunked", seed=3)
MLA = KVConfig("mla", layers=61, planes=1, block_tokens=64, row_bytes=576 * 2, dtype="bf16",
               programs=256, ctx_kind="lognormal", ctx_median=8192, ctx_lo=1024, ctx_hi=32768,
               busy_frac=0.5, gpu_pct=40.0, frag="chunked", seed=4)
CHURN = KVConfig("churn", layers=32, planes=2, block_tokens=16, row_bytes=8 * 128 * 2, dtype="bf16",
                 programs=1024, ctx_kind="lognormal", ctx_median=4096, ctx_lo=512, ctx_hi=32768,
                 busy_frac=0.5, gpu_pct=55.0, frag="shuffled", seed=5, steps=100, flip_frac=0.1,
                 pct_swing=(55.0, 10.0))

CONFIGS = {c.name: c for c in (TINY, LLAMA3_8B, LLAMA3_70B, LLAMA3_70B_TP2, LLAMA3_70B_TP4, LLAMA3_70B_TP8, MLA,
                                CHURN)}
