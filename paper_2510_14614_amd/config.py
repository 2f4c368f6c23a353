"""Model configuration for the FAL / FAL+ / GPT training step.

The fields mirror ``fal_config_t`` in ``include/fal.h`` one to one.  The
architectures are the Pre-LN GPT block (Sec. 2, Eq. 1), the FAL block
(Sec. 4.1, Eq. 2), the FAL+ block (Sec. 5; Appendix D equations) and the
parallel configuration the paper compares against in Sec. 6.1 and 6.4
(MHA and MLP read the same block input).
"""
from __future__ import annotations

import dataclasses

ARCH_GPT, ARCH_FAL, ARCH_FALPLUS, ARCH_PARALLEL = 0, 1, 2, 3
ARCH_NAMES = {"gpt": ARCH_GPT, "fal": ARCH_FAL, "falplus": ARCH_FALPLUS, "fal+": ARCH_FALPLUS,
              "parallel": ARCH_PARALLEL}
DTYPE_F32, DTYPE_BF16 = 0, 1
SCHED_SEQ, SCHED_STREAMS, SCHED_MERGED, SCHED_STREAMS_MERGED = 0, 1, 2, 3
SCHED_NAMES = {"seq": SCHED_SEQ, "streams": SCHED_STREAMS, "merged": SCHED_MERGED,
               "streams_merged": SCHED_STREAMS_MERGED}


@dataclasses.dataclass
class Config:
    n_layer: int
    d_model: int
    n_head: int          # heads held on this GPU (all heads unless a shard)
    head_dim: int
    d_ff: int
    vocab: int
    seq_len: int
    batch: int
    arch: int = ARCH_FAL
    dtype: int = DTYPE_F32
    sched: int = SCHED_SEQ
    ln_eps: float = 1e-5
    gelu_tanh: int = 1        # 1: tanh approximation, 0: erf form
    has_embed_head: int = 1   # 0: block stack only (no embedding, no LM head)
    fal_block1_mode: int = 0  # FAL only: 0 Eq. 2 in block 1 too, 1 standard block 1 emitting F
    bidirectional: int = 0    # 1: no attention mask (encoder blocks; block stack only)
    n_kv_head: int = 0        # key/value heads (grouped-query attention); 0: n_head

    @property
    def kv_heads(self) -> int:
        return self.n_kv_head or self.n_head

    @property
    def d_kv(self) -> int:
        return self.kv_heads * self.head_dim

    @property
    def d_qkv(self) -> int:
        return self.d_attn + 2 * self.d_kv

    @property
    def d_attn(self) -> int:
        return self.n_head * self.head_dim

    @property
    def tokens(self) -> int:
        return self.batch * self.seq_len

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)

    def train_flops_per_token(self) -> float:
        """Algorithmic training FLOPs per token: forward+backward counted as
        three forwards, causal attention at (T+1)/2 keys per query (T keys
        when bidirectional), tied head."""
        d, dA, f, T, V = self.d_model, self.d_attn, self.d_ff, self.seq_len, self.vocab
        # QK^T and PV: 4 dA FLOPs per (query, key); (T+1)/2 keys per query
        # under the causal mask, T without it
        keys = 2 * T if self.bidirectional else T + 1
        per_layer = 2 * d * self.d_qkv + 2 * dA * d + 4 * d * f + 2 * dA * keys
        head = 2 * d * V if self.has_embed_head else 0
        return 3.0 * (self.n_layer * per_layer + head)


# The workload shapes: a tiny fp32 model, GPT-2-small and GPT-2-medium
# shaped models, a ~1.3B GPT shape, one GPU's tensor-parallel share of a
# ~7B block stack (8 of 32 heads, FFN 11008/4), and the 48-block encoder
# stack of the masked-language-model depth study (BERT-Large blocks, no
# attention mask, sequence 128; one micro-batch of 128 sequences), also with
# grouped-query attention in two groups as in the transformer-variant study.
CONFIGS = {
    "tiny": Config(n_layer=2, d_model=64, n_head=4, head_dim=16, d_ff=256, vocab=256,
                   seq_len=32, batch=2, arch=ARCH_FAL, dtype=DTYPE_F32),
    "gpt2-small": Config(n_layer=12, d_model=768, n_head=12, head_dim=64, d_ff=3072,
                         vocab=50257, seq_len=1024, batch=8, arch=ARCH_FAL, dtype=DTYPE_BF16),
    "gpt2-medium": Config(n_layer=24, d_model=1024, n_head=16, head_dim=64, d_ff=4096,
                          vocab=50257, seq_len=1024, batch=8, arch=ARCH_FALPLUS, dtype=DTYPE_BF16),
    "gpt-1.3b": Config(n_layer=24, d_model=2048, n_head=16, head_dim=128, d_ff=8192,
                       vocab=50257, seq_len=2048, batch=4, arch=ARCH_FAL, dtype=DTYPE_BF16),
    "7b-tp-shard": Config(n_layer=32, d_model=4096, n_head=8, head_dim=128, d_ff=2752,
                          vocab=0, seq_len=2048, batch=2, arch=ARCH_FAL, dtype=DTYPE_BF16,
                          has_embed_head=0),
    "mlm-48": Config(n_layer=48, d_model=1024, n_head=16, head_dim=64, d_ff=4096, vocab=0, seq_len=128,
                     batch=128, arch=ARCH_FAL, dtype=DTYPE_BF16, has_embed_head=0, bidirectional=1),
    "mlm-48-gqa2": Config(n_layer=48, d_model=1024, n_head=16, head_dim=64, d_ff=4096, vocab=0, seq_len=128,
                          batch=128, arch=ARCH_FAL, dtype=DTYPE_BF16, has_embed_head=0, bidirectional=1,
                          n_kv_head=2),
}


def get_config(name: str, **overrides) -> Config:
    return dataclasses.replace(CONFIGS[name], **overrides)
