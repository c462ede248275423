"""Configuration presets for the Domino drafter.

Dimensions follow the Qwen3 target shapes named by the workloads; the Domino
head sizes (GRU width 1024, low-rank width 256, block 16, 5 backbone layers)
are the ones the paper's implementation details give (Sec. 5.1).
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class DominoConfig:
    name: str
    hidden: int            # d: drafter / target hidden width
    n_layers: int          # backbone depth
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int               # SwiGLU intermediate width
    vocab: int             # V
    block: int = 16        # B: anchor + B-1 draft positions
    gru_hidden: int = 1024  # d_s
    rank: int = 256        # r
    mask_token_id: int = -1  # -1 means vocab-1
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    dtype: str = "bf16"    # storage type of weights and KV: "bf16" or "f32"
    # workload
    batch: int = 1
    ctx: int = 1024
    branch: int = 1        # beta: top-k per position used by the tree
    ctx_from_hidden: bool = False  # context KV built by projecting hidden states
    # k > 0: a context row is the concatenation of k target layers' hidden
    # states ([k*d]), fused to width d by ctx_fc before the K/V projections
    ctx_fuse_layers: int = 0

    @property
    def mask_id(self) -> int:
        return self.vocab - 1 if self.mask_token_id < 0 else self.mask_token_id

    @property
    def ctx_width(self) -> int:
        """Width of one target-hidden-state context row."""
        return self.hidden * self.ctx_fuse_layers if self.ctx_fuse_layers > 0 else self.hidden

    @property
    def depth(self) -> int:
        return self.block - 1

    @property
    def n_nodes(self) -> int:
        return 1 + self.depth * self.branch

    def with_(self, **kw) -> "DominoConfig":
        return replace(self, **kw)


PRESETS = {
    # tiny fp32 drafter; context comes from N(0,1) target hidden states
    "tiny": DominoConfig("tiny", hidden=256, n_layers=2, n_q_heads=4, n_kv_heads=2,
                         head_dim=64, ffn=1024, vocab=4096, dtype="f32", batch=1,
                         ctx=128, branch=1, ctx_from_hidden=True),
    # Qwen3-8B-shaped bf16 drafter, bs 1, ctx 1024 (latency setting)
    "qwen3_8b": DominoConfig("qwen3_8b", hidden=4096, n_layers=5, n_q_heads=32,
                             n_kv_heads=8, head_dim=128, ffn=12288, vocab=151936,
                             batch=1, ctx=1024, branch=1, ctx_fuse_layers=5),
    # serving-style: bs 32, ctx 2048, tree branch 4
    "qwen3_8b_bs32": DominoConfig("qwen3_8b_bs32", hidden=4096, n_layers=5, n_q_heads=32,
                                  n_kv_heads=8, head_dim=128, ffn=12288, vocab=151936,
                                  batch=32, ctx=2048, branch=4, ctx_fuse_layers=5),
    # Qwen3-4B-shaped, long context
    "qwen3_4b_ctx8k": DominoConfig("qwen3_4b_ctx8k", hidden=2560, n_layers=5, n_q_heads=32,
                                   n_kv_heads=8, head_dim=128, ffn=9728, vocab=151936,
                                   batch=4, ctx=8192, branch=1, ctx_fuse_layers=5),
    # Qwen3-32B-shaped
    "qwen3_32b": DominoConfig("qwen3_32b", hidden=5120, n_layers=5, n_q_heads=64,
                              n_kv_heads=8, head_dim=128, ffn=25600, vocab=151936,
                              batch=16, ctx=4096, branch=1, ctx_fuse_layers=5),
    # target models (the verify forward): a small fp32 decoder sharing the tiny
    # drafter's vocabulary and width, and the Qwen3-8B-shaped target (36 layers)
    "tiny_target": DominoConfig("tiny_target", hidden=256, n_layers=4, n_q_heads=4, n_kv_heads=2,
                                head_dim=64, ffn=1024, vocab=4096, dtype="f32", batch=1, ctx=128),
    "qwen3_8b_target": DominoConfig("qwen3_8b_target", hidden=4096, n_layers=36, n_q_heads=32,
                                    n_kv_heads=8, head_dim=128, ffn=12288, vocab=151936,
                                    batch=1, ctx=1024, branch=1),
}


def get_config(name: str, **overrides) -> DominoConfig:
    cfg = PRESETS[name]
    return cfg.with_(**overrides) if overrides else cfg
