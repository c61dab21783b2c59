"""Seeded synthetic inputs shared by the HIP path's tests, the oracle's tests and the benchmark.

This module holds shapes and random draws only: it computes no step of the method.  Every
tensor is drawn from a NumPy ``default_rng`` seeded by (base seed, tensor name), so any
subset of a model's tensors can be regenerated on its own.  Float tensors are rounded once
to bfloat16 (round to nearest even) and returned as float32 arrays holding exactly those
bfloat16 values, so the HIP path (which stores them as bf16) and the oracle (which reads
them as float64) see identical numbers.

Model shapes follow the three workloads the method is evaluated on: a small tiny stack used
for exact parity, a 32-layer ViT with 2x2 patch merge in front of a 28-layer GQA decoder,
and the screenshot size of the agent traces.  The paper's own model (a 64-layer ViT and a
40-layer LLM, Sec. 5.1) and dataset are not available; these synthetic stand-ins carry
their structure: pre-LN ViT with bidirectional attention, an adapter that merges 2x2
patches into the LLM width, and a RoPE/GQA/SwiGLU decoder with a paged KV cache.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import numpy as np


# --------------------------------------------------------------------------------------
# shapes
# --------------------------------------------------------------------------------------
@dataclass(frozen=True)
class VitConfig:
    hidden: int
    heads: int
    mlp: int
    layers: int
    patch: int
    merge: int          # 1: no merge (adapter is LN + Linear); 2: 2x2 patch merge
    out_hidden: int     # LLM hidden size the adapter projects to
    image_h: int
    image_w: int
    channels: int = 3
    eps: float = 1e-6
    name: str = "vit"

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def grid_h(self) -> int:
        return self.image_h // self.patch

    @property
    def grid_w(self) -> int:
        return self.image_w // self.patch

    @property
    def n_patches(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def n_out(self) -> int:
        return self.n_patches // (self.merge * self.merge)

    @property
    def patch_dim(self) -> int:
        return self.channels * self.patch * self.patch


@dataclass(frozen=True)
class LlmConfig:
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    inter: int
    vocab: int
    layers: int
    rope_theta: float = 10000.0
    eps: float = 1e-6
    block: int = 16     # tokens per paged-KV block
    name: str = "llm"


# Tiny stack: exact-parity workload (fp32 oracle vs bf16 GPU), image 32x32x3, patch 4.
TINY_VIT = VitConfig(hidden=256, heads=4, mlp=1024, layers=1, patch=4, merge=1, out_hidden=256,
                     image_h=32, image_w=32, name="tiny_vit")
TINY_LLM = LlmConfig(hidden=256, n_q=4, n_kv=2, head_dim=64, inter=688, vocab=4096, layers=2,
                     name="tiny_llm")
TINY_TEXT = 32          # text tokens after the 64 vision tokens
TINY_DECODE_STEPS = 16

# Vision encoder at real width: 1008x1008 image, patch 14 -> 72x72 = 5184 patches -> 1296 merged.
VIT_1008 = VitConfig(hidden=1280, heads=16, mlp=5120, layers=32, patch=14, merge=2, out_hidden=3584,
                     image_h=1008, image_w=1008, name="vit32_1008")
# The same encoder on a 1092x2408 screenshot: 78x172 = 13416 patches -> 3354 merged tokens.
VIT_SCREEN = VitConfig(hidden=1280, heads=16, mlp=5120, layers=32, patch=14, merge=2, out_hidden=3584,
                       image_h=1092, image_w=2408, name="vit32_screen")
# Decoder at real width: 28 layers, 28 q / 4 kv heads of 128, SwiGLU 18944, vocab 152064.
LLM_28 = LlmConfig(hidden=3584, n_q=28, n_kv=4, head_dim=128, inter=18944, vocab=152064, layers=28,
                   name="llm28")
LLM_VISION_TOKENS = 1300
LLM_TEXT_TOKENS = 200
LLM_DECODE_STEPS = 64


# --------------------------------------------------------------------------------------
# random draws
# --------------------------------------------------------------------------------------
def _rng(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([seed, zlib.crc32(name.encode())])


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = (u + (((u >> 16) & 1) + np.uint32(0x7FFF))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def normal(shape, seed: int, name: str, std: float = 0.02, mean: float = 0.0) -> np.ndarray:
    r = _rng(seed, name).standard_normal(size=shape, dtype=np.float32)
    return bf16_round(r * np.float32(std) + np.float32(mean))


def vit_layer_names(l: int) -> list[str]:
    p = f"l{l}."
    return [p + s for s in ("ln1.g", "ln1.b", "qkv.w", "qkv.b", "o.w", "o.b",
                            "ln2.g", "ln2.b", "fc1.w", "fc1.b", "fc2.w", "fc2.b")]


def vit_shapes(cfg: VitConfig) -> dict[str, tuple]:
    H, I = cfg.hidden, cfg.mlp
    s = {"patch.w": (H, cfg.patch_dim), "patch.b": (H,), "pos": (cfg.n_patches, H)}
    for l in range(cfg.layers):
        p = f"l{l}."
        s.update({p + "ln1.g": (H,), p + "ln1.b": (H,), p + "qkv.w": (3 * H, H), p + "qkv.b": (3 * H,),
                  p + "o.w": (H, H), p + "o.b": (H,), p + "ln2.g": (H,), p + "ln2.b": (H,),
                  p + "fc1.w": (I, H), p + "fc1.b": (I,), p + "fc2.w": (H, I), p + "fc2.b": (H,)})
    m2 = cfg.merge * cfg.merge
    s.update({"merge.ln.g": (H,), "merge.ln.b": (H,), "merge.w": (cfg.out_hidden, m2 * H),
              "merge.b": (cfg.out_hidden,)})
    return s


def llm_shapes(cfg: LlmConfig) -> dict[str, tuple]:
    H, d, I = cfg.hidden, cfg.head_dim, cfg.inter
    s = {"embed": (cfg.vocab, H)}
    for l in range(cfg.layers):
        p = f"l{l}."
        s.update({p + "rms1.g": (H,), p + "q.w": (cfg.n_q * d, H), p + "k.w": (cfg.n_kv * d, H),
                  p + "v.w": (cfg.n_kv * d, H), p + "o.w": (H, cfg.n_q * d), p + "rms2.g": (H,),
                  p + "gate.w": (I, H), p + "up.w": (I, H), p + "down.w": (H, I)})
    s.update({"norm.g": (H,), "lm_head.w": (cfg.vocab, H)})
    return s


def _draw(name: str, shape: tuple, seed: int) -> np.ndarray:
    # Norm gains near 1 and norm shifts away from 0, so that a dropped affine term shows up.
    if name.endswith(".g"):
        return normal(shape, seed, name, std=0.2, mean=1.0)
    if name.endswith("ln1.b") or name.endswith("ln2.b") or name.endswith("ln.b"):
        return normal(shape, seed, name, std=0.2)
    return normal(shape, seed, name, std=0.02)


def vit_weights(cfg: VitConfig, seed: int = 0, names=None) -> dict[str, np.ndarray]:
    shapes = vit_shapes(cfg)
    keys = shapes.keys() if names is None else names
    return {k: _draw(k, shapes[k], seed) for k in keys}


def llm_weights(cfg: LlmConfig, seed: int = 0, names=None) -> dict[str, np.ndarray]:
    shapes = llm_shapes(cfg)
    keys = shapes.keys() if names is None else names
    return {k: _draw(k, shapes[k], seed) for k in keys}


def _draw_torch(name: str, shape: tuple, seed: int, device):
    """The same distributions as _draw, drawn on `device` by torch's generator (seeded per tensor
    name) and rounded to bf16: full-size models are generated in seconds rather than minutes.
    The values differ from _draw's (another generator); each caller uses one source for both the
    library and the oracle."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) << 32) | zlib.crc32(name.encode()))
    std, mean = 0.02, 0.0
    if name.endswith(".g"):
        std, mean = 0.2, 1.0
    elif name.endswith("ln1.b") or name.endswith("ln2.b") or name.endswith("ln.b"):
        std = 0.2
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return (t * std + mean).to(torch.bfloat16)


def vit_weights_torch(cfg: VitConfig, seed: int = 0, device="cuda") -> dict:
    """vit_weights' tensors as bf16 torch tensors drawn on `device`."""
    return {k: _draw_torch(k, v, seed, device) for k, v in vit_shapes(cfg).items()}


def llm_weights_torch(cfg: LlmConfig, seed: int = 0, device="cuda") -> dict:
    """llm_weights' tensors as bf16 torch tensors drawn on `device`."""
    return {k: _draw_torch(k, v, seed, device) for k, v in llm_shapes(cfg).items()}


def to_host(weights: dict) -> dict[str, np.ndarray]:
    """Host float32 copies (bf16-exact values) of a dict of bf16 torch tensors."""
    return {k: v.float().cpu().numpy() for k, v in weights.items()}


def image(batch: int, h: int, w: int, seed: int = 1, channels: int = 3) -> np.ndarray:
    """Uniform[0,1) pixels, HWC, rounded to bf16: [batch, h, w, channels] float32."""
    r = _rng(seed, f"image{batch}x{h}x{w}").random(size=(batch, h, w, channels), dtype=np.float32)
    return bf16_round(r)


def text_ids(n: int, vocab: int, seed: int = 2) -> np.ndarray:
    return _rng(seed, f"ids{n}").integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def vision_embeds(n: int, hidden: int, seed: int = 4) -> np.ndarray:
    """Stand-in for adapter output when the LLM is run alone: N(0, 0.02) rounded to bf16."""
    return normal((n, hidden), seed, f"visemb{n}", std=0.02)


def block_tables(lengths, block: int, seed: int = 5, num_blocks: int | None = None,
                 shuffle: bool = True) -> tuple[np.ndarray, int]:
    """Assign disjoint physical KV blocks to each sequence.

    ``lengths[b]`` is the largest number of tokens sequence b will hold.  Returns an int32
    table ``[B, max_blocks]`` (unused entries are -1) and the pool size in blocks.  With
    ``shuffle`` the physical ids are a random permutation, so that a kernel which assumes
    contiguous blocks fails.
    """
    need = [(int(n) + block - 1) // block for n in lengths]
    total = sum(need)
    pool = total if num_blocks is None else int(num_blocks)
    if pool < total:
        raise ValueError("pool too small")
    ids = np.arange(pool, dtype=np.int64)
    if shuffle:
        ids = _rng(seed, f"blocks{pool}").permutation(pool)
    maxb = max(need) if need else 0
    table = np.full((len(need), max(maxb, 1)), -1, dtype=np.int32)
    o = 0
    for b, nb in enumerate(need):
        table[b, :nb] = ids[o:o + nb]
        o += nb
    return table, pool
