"""Model shapes and synthetic workloads.

The five workloads are the paper-shaped benchmark cases: a tiny parity model,
a 4B-class dense decoder at batch 1 and batch 32, a 9B-class decoder at batch
8, and a prefill-dominated 4B-class long-prompt run.  Shapes only: no method
arithmetic lives here.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_base: float = 1e6
    rms_eps: float = 1e-6
    gain_mode: int = 0          # 0: RMSNorm gains are 1; 1: 1 + 10*R-spec
    heads: int = 0              # paper-default heads (HEADS_* flags); 0: the one-linear forms

    @property
    def pad_id(self) -> int:
        """The reserved PAD token: the last vocabulary row."""
        return self.vocab - 1

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n: int) -> "ModelConfig":
        return replace(self, n_layers=n)

    def layer_params(self) -> int:
        h, f = self.hidden, self.ffn
        return h * (self.q_dim + 2 * self.kv_dim) + self.q_dim * h + 3 * h * f

    def weight_bytes_bf16(self) -> int:
        """bf16 bytes of every matrix (E counted once)."""
        h = self.hidden
        return 2 * (self.n_layers * self.layer_params() + self.vocab * h + 2 * (h * 2 * h))

    def kv_bytes_per_latent(self) -> int:
        return 2 * self.n_layers * self.kv_dim * 2


#: ``ModelConfig.heads`` flags: the App. B forms of the three heads.
HEADS_MLP_COMPRESSOR = 1     # z = E[a] + E[b] + W2 SiLU(W1 [E[a]; E[b]])  (Table 4, MLP)
HEADS_MTP_LAYER = 2          # h_d = Layer(W_fc [...]) with its own latent KV cache (App. B.2)
HEADS_MLP_CONFIDENCE = 4     # c = sigmoid(W2 SiLU(W1 RMSNorm([h_b; h_d])))  (App. B.3)
HEADS_PAPER = 7


def model_tensor_shapes(cfg: ModelConfig) -> dict:
    """Logical ``[out][in]`` shapes of every tensor, keyed by name."""
    h = cfg.hidden
    shapes = {
        "embed": (cfg.vocab, h), "w_comp": (h, 2 * h), "b_comp": (h,),
        "w_fc": (h, 2 * h), "w_conf": (2 * h,),
        "g_final": (h,), "g_mtp_h": (h,), "g_mtp_e": (h,), "g_mtp_o": (h,),
        "g_conf": (2 * h,),
    }
    for li in range(cfg.n_layers):
        shapes[f"l{li}.wq"] = (cfg.q_dim, h)
        shapes[f"l{li}.wk"] = (cfg.kv_dim, h)
        shapes[f"l{li}.wv"] = (cfg.kv_dim, h)
        shapes[f"l{li}.wo"] = (h, cfg.q_dim)
        shapes[f"l{li}.wgate"] = (cfg.ffn, h)
        shapes[f"l{li}.wup"] = (cfg.ffn, h)
        shapes[f"l{li}.wdown"] = (h, cfg.ffn)
        shapes[f"l{li}.g_attn"] = (h,)
        shapes[f"l{li}.g_ffn"] = (h,)
    if cfg.heads & HEADS_MLP_COMPRESSOR:
        shapes["comp_w1"] = (h, 2 * h)
        shapes["comp_w2"] = (h, h)
    if cfg.heads & HEADS_MTP_LAYER:
        for name, shp in (("wq", (cfg.q_dim, h)), ("wk", (cfg.kv_dim, h)), ("wv", (cfg.kv_dim, h)),
                          ("wo", (h, cfg.q_dim)), ("wgate", (cfg.ffn, h)), ("wup", (cfg.ffn, h)),
                          ("wdown", (h, cfg.ffn)), ("g_attn", (h,)), ("g_ffn", (h,))):
            shapes[f"mtp.{name}"] = shp
    if cfg.heads & HEADS_MLP_CONFIDENCE:
        shapes["conf_w1"] = (h, 2 * h)
        shapes["conf_w2"] = (h,)
    return shapes


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    prompt_tokens: int
    decode_steps: int
    tau: float
    temperature: float = 0.0     # <= 0: greedy
    top_p: float = 1.0
    top_k: int = 0               # evaluation sampler (Sec. 4): 0 = off
    rep_penalty: float = 1.0     # evaluation sampler: 1 = off
    prefill_chunk: int = 4096    # latent positions per prefill chunk
    weight_precision: str = "bf16"   # precision of the stored weights
    seed: int = 0
    prompt_seed: int = 1
    sample_seed_base: int = 1000
    notes: str = field(default="", compare=False)

    @property
    def latents(self) -> int:
        return (self.prompt_tokens + 1) // 2

    @property
    def max_latent(self) -> int:
        return self.latents + self.decode_steps


TINY = ModelConfig(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                   ffn=1024, vocab=4096, rope_base=1e4, rms_eps=1e-6)
DENSE_4B = ModelConfig(n_layers=36, hidden=2560, n_q_heads=32, n_kv_heads=8,
                       head_dim=128, ffn=9728, vocab=151936, rope_base=1e6, rms_eps=1e-6)
DENSE_9B = ModelConfig(n_layers=32, hidden=4096, n_q_heads=32, n_kv_heads=8,
                       head_dim=128, ffn=12288, vocab=151936, rope_base=1e6, rms_eps=1e-6)

WORKLOADS = {
    # tiny 2-layer decoder, fp32 weights, 64-token prompt, 16 greedy pair steps
    "tiny-bs1": Workload("tiny-bs1", TINY, batch=1, prompt_tokens=64, decode_steps=16,
                         tau=0.5, weight_precision="fp32"),
    # 4B-class, batch 1, 4096-token prompt (2048 latents), 256 greedy pair steps
    "4b-bs1-ctx2048": Workload("4b-bs1-ctx2048", DENSE_4B, batch=1, prompt_tokens=4096,
                               decode_steps=256, tau=0.95),
    # 4B-class, batch 32, 16384-token prompts, top-p 0.95 at T 0.6, tau 0.7
    "4b-bs32-ctx8192-topp": Workload("4b-bs32-ctx8192-topp", DENSE_4B, batch=32,
                                     prompt_tokens=16384, decode_steps=128, tau=0.7,
                                     temperature=0.6, top_p=0.95),
    # 9B-class, batch 8, 32768-token prompts, greedy
    "9b-bs8-ctx16384": Workload("9b-bs8-ctx16384", DENSE_9B, batch=8, prompt_tokens=32768,
                                decode_steps=128, tau=0.95),
    # 4B-class prefill of a 65536-token prompt in 4096-latent chunks, then 64 steps
    "4b-prefill-ctx32768": Workload("4b-prefill-ctx32768", DENSE_4B, batch=1,
                                    prompt_tokens=65536, decode_steps=64, tau=0.5),
}
