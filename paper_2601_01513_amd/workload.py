"""Seeded synthetic workloads for the verifier scoring pass.

This module holds the workload shapes and the seeded random inputs that both
the HIP path and the CPU oracle consume. It contains none of the method's
arithmetic: only shapes, random draws and dtype rounding of those draws.

The workloads stand in for the paper's video-QA inputs (VideoSimpleQA,
EncVQA; Section 4.1), which are not available: a verifier decoder shaped like
the paper's verifiers (Qwen2.5-VL 7B/32B class, Section 4.3), random-init
weights, a prefix of visual-frame rows followed by text ids (retrieved
passages plus the question, Eq. 4 and Eq. 6 conditioning on (Q, V)), and M
drafted candidates (Eq. 5 and Eq. 8-10 produce them; here they are uniform
random ids).

Recipe (every tensor has its own seed derived from (seed, tensor name)):
  * weight matrices, embedding and LM head: N(0, 0.02), drawn in fp32 and
    rounded to bf16 (round-to-nearest-even) for bf16 workloads;
  * RMSNorm gains: 1.0;
  * visual rows: N(0, 1) * 0.02, rounded like the weights;
  * prefix text ids and candidate ids: uniform over [0, vocab);
  * candidate lengths: Cmax for every candidate, or uniform over
    [lo, hi] inclusive for ragged workloads; positions past a candidate's
    length hold pad id 0.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F32 = 0
BF16 = 1


@dataclasses.dataclass(frozen=True)
class VerifierConfig:
    """Shape of one verifier workload (decoder + prefix + candidates)."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_base: float
    dtype: int  # F32 or BF16
    n_prefix: int  # P = visual rows + text ids
    n_visual: int  # Pv
    n_cands: int  # M
    cand_len: int  # Cmax
    ragged: Optional[Tuple[int, int]] = None  # inclusive length range
    rms_eps: float = 1e-6

    @property
    def n_text(self) -> int:
        return self.n_prefix - self.n_visual

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def n_params(self) -> int:
        d, L = self.d_model, self.n_layers
        per_layer = (2 * d + self.qkv_rows * d + d * self.n_heads * self.head_dim
                     + 2 * self.d_ff * d + d * self.d_ff)
        return 2 * self.vocab * d + d + L * per_layer

    def replace(self, **kw) -> "VerifierConfig":
        return dataclasses.replace(self, **kw)


# The five workloads of the scoring pass, named by what they are.
TINY_F32 = VerifierConfig(
    name="tiny-fp32 L2 d256 P256 M4x32", n_layers=2, d_model=256, n_heads=4,
    n_kv_heads=4, head_dim=64, d_ff=704, vocab=4096, rope_base=10000.0,
    dtype=F32, n_prefix=256, n_visual=64, n_cands=4, cand_len=32)
B1_5 = VerifierConfig(
    name="1.5B-class bf16 P2048 M4x64", n_layers=28, d_model=1536, n_heads=12,
    n_kv_heads=2, head_dim=128, d_ff=8960, vocab=151936, rope_base=1e6,
    dtype=BF16, n_prefix=2048, n_visual=1024, n_cands=4, cand_len=64)
B7 = VerifierConfig(
    name="7B-class bf16 P4096 M8x64", n_layers=28, d_model=3584, n_heads=28,
    n_kv_heads=4, head_dim=128, d_ff=18944, vocab=152064, rope_base=1e6,
    dtype=BF16, n_prefix=4096, n_visual=2048, n_cands=8, cand_len=64)
B7_LONG = B7.replace(
    name="7B-class bf16 P16384 M16x<=128 ragged", n_prefix=16384,
    n_visual=8192, n_cands=16, cand_len=128, ragged=(32, 128))
B32 = VerifierConfig(
    name="32B-class bf16 P8192 M16x128", n_layers=64, d_model=5120,
    n_heads=40, n_kv_heads=8, head_dim=128, d_ff=27648, vocab=152064,
    rope_base=1e6, dtype=BF16, n_prefix=8192, n_visual=4096, n_cands=16,
    cand_len=128)

CONFIGS: List[VerifierConfig] = [TINY_F32, B1_5, B7, B7_LONG, B32]

# Drafting (Eq. 5, 8-10): a 3B-class drafter (36 layers, d 2048, 16/2 heads,
# d_ff 11008) continues k = 3 branches, one per retrieved document, after the
# shared (visual, question) prefix: 2048 visual rows + 128 question tokens,
# each branch prompt a 512-token document plus its generation prompt, 64 new
# tokens per branch (the entity, reasoning and answer generations together).
DRAFT_3B = VerifierConfig(
    name="3B-class drafter bf16 P2176 3 branches x 512 + 64 new", n_layers=36, d_model=2048,
    n_heads=16, n_kv_heads=2, head_dim=128, d_ff=11008, vocab=151936, rope_base=1e6,
    dtype=BF16, n_prefix=2176, n_visual=2048, n_cands=3, cand_len=512)
DRAFT_NEW = 64
HEADLINE = B7


def tensor_seed(seed: int, name: str) -> int:
    """Stable per-tensor seed from (workload seed, tensor name)."""
    return (zlib.crc32(f"{seed}:{name}".encode()) << 16) ^ (seed & 0xFFFF)


def host_rng(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([seed, zlib.crc32(name.encode())])


def cand_lengths(cfg: VerifierConfig, seed: int) -> np.ndarray:
    if cfg.ragged is None:
        return np.full(cfg.n_cands, cfg.cand_len, dtype=np.int32)
    lo, hi = cfg.ragged
    return host_rng(seed, "cand_len").integers(
        lo, hi + 1, size=cfg.n_cands).astype(np.int32)


def make_ids(cfg: VerifierConfig, seed: int):
    """Prefix text ids [P - Pv], candidate ids [M][Cmax] (pad 0), lengths [M]."""
    prefix_ids = host_rng(seed, "prefix_ids").integers(
        0, cfg.vocab, size=cfg.n_text).astype(np.int32)
    cand_ids = host_rng(seed, "cand_ids").integers(
        0, cfg.vocab, size=(cfg.n_cands, cfg.cand_len)).astype(np.int32)
    lens = cand_lengths(cfg, seed)
    for m in range(cfg.n_cands):
        cand_ids[m, lens[m]:] = 0
    return prefix_ids, cand_ids, lens


def _torch():
    import torch
    return torch


def _normal(shape, std, seed, name, device, dtype):
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(tensor_seed(seed, name))
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    t.mul_(std)
    return t.to(dtype)


def torch_dtype(cfg: VerifierConfig):
    torch = _torch()
    return torch.float32 if cfg.dtype == F32 else torch.bfloat16


def make_weights(cfg: VerifierConfig, seed: int, device="cpu") -> Dict:
    """Random-init decoder weights as torch tensors on `device`.

    Layout is the torch nn.Linear layout [out][in]:
      embed, lm_head [V][d]; final_norm [d];
      per layer: attn_norm [d], wqkv [(Hq+2Hkv)*hd][d] (q rows, then k rows,
      then v rows, head-major), wo [d][Hq*hd], ffn_norm [d],
      wgu [2F][d] (gate rows, then up rows), wdown [d][F].
    """
    torch = _torch()
    dt = torch_dtype(cfg)
    d = cfg.d_model
    ones = lambda: torch.ones(d, device=device, dtype=dt)  # noqa: E731
    w = {
        "embed": _normal((cfg.vocab, d), 0.02, seed, "embed", device, dt),
        "lm_head": _normal((cfg.vocab, d), 0.02, seed, "lm_head", device, dt),
        "final_norm": ones(),
        "layers": [],
    }
    for i in range(cfg.n_layers):
        w["layers"].append({
            "attn_norm": ones(),
            "wqkv": _normal((cfg.qkv_rows, d), 0.02, seed, f"l{i}.wqkv", device, dt),
            "wo": _normal((d, cfg.n_heads * cfg.head_dim), 0.02, seed, f"l{i}.wo", device, dt),
            "ffn_norm": ones(),
            "wgu": _normal((2 * cfg.d_ff, d), 0.02, seed, f"l{i}.wgu", device, dt),
            "wdown": _normal((d, cfg.d_ff), 0.02, seed, f"l{i}.wdown", device, dt),
        })
    return w


def make_visual(cfg: VerifierConfig, seed: int, device="cpu"):
    return _normal((cfg.n_visual, cfg.d_model), 0.02, seed, "visual", device,
                   torch_dtype(cfg))


@dataclasses.dataclass
class Workload:
    cfg: VerifierConfig
    seed: int
    weights: Dict
    visual: object  # torch tensor [Pv][d]
    prefix_ids: np.ndarray
    cand_ids: np.ndarray
    cand_len: np.ndarray


def make_workload(cfg: VerifierConfig, seed: int, device="cpu") -> Workload:
    prefix_ids, cand_ids, lens = make_ids(cfg, seed)
    return Workload(cfg, seed, make_weights(cfg, seed, device),
                    make_visual(cfg, seed, device), prefix_ids, cand_ids, lens)


def input_fingerprint(wl: Workload, samples: int = 4096) -> str:
    """SHA-256 over the exact bits of the ids and lengths and of an evenly
    strided sample of every weight tensor and of the visual rows: names the
    generated inputs without copying them all to the host."""
    import hashlib
    torch = _torch()
    h = hashlib.sha256()
    for a in (wl.prefix_ids, wl.cand_ids, wl.cand_len):
        h.update(np.ascontiguousarray(a).tobytes())
    tensors = [wl.weights["embed"], wl.weights["lm_head"], wl.weights["final_norm"], wl.visual]
    for lw in wl.weights["layers"]:
        tensors += [lw[k] for k in sorted(lw)]
    for t in tensors:
        flat = t.detach().reshape(-1)
        step = max(1, flat.numel() // samples)
        s = flat[::step][:samples].contiguous()
        bits = s.view(torch.int16) if s.element_size() == 2 else s.view(torch.int32)
        h.update(bits.cpu().numpy().tobytes())
    return h.hexdigest()


def to_host_f32(t) -> np.ndarray:
    """Exact host copy of a (bf16 or fp32) tensor as float32."""
    return t.detach().float().cpu().numpy()


class HostLayers(Sequence):
    """Per-layer host copies of device weights, fetched on access."""

    def __init__(self, layers: List[Dict]):
        self._layers = layers

    def __len__(self):
        return len(self._layers)

    def __getitem__(self, i):
        if isinstance(i, slice):
            return [self[j] for j in range(*i.indices(len(self)))]
        return {k: to_host_f32(v) for k, v in self._layers[i].items()}


def host_weights(weights: Dict, lazy: bool = False) -> Dict:
    """Host (numpy float32) view of `make_weights` output for the oracle."""
    layers = HostLayers(weights["layers"])
    return {
        "embed": to_host_f32(weights["embed"]),
        "lm_head": to_host_f32(weights["lm_head"]),
        "final_norm": to_host_f32(weights["final_norm"]),
        "layers": layers if lazy else list(layers),
    }


# ------------------------------------------------------- retrieval-stage inputs
# Stand-ins for a short video and a CLIP embedding bank (the paper's videos
# last about 22 s; CLIP ViT-L/14-336 embeds frames of 336 x 336 into 768
# dimensions). No arithmetic of the method happens here.

@dataclasses.dataclass(frozen=True)
class RetrievalConfig:
    name: str
    n_frames: int      # decoded frames of the video
    height: int
    width: int
    n_scenes: int      # the video cuts between this many scenes
    n_docs: int        # document embeddings in the bank
    dim: int           # embedding width
    k: int             # documents retrieved per keyframe
    K: int             # documents kept in T*
    theta: float       # keyframe threshold on the histogram similarity


VIDEO_SMALL = RetrievalConfig("small video 40x24x32, 5 scenes, 300 docs", 40, 24, 32, 5, 300,
                              64, 3, 3, 0.6)
# About 22 s at 10 frames/s, CLIP-sized frames and embeddings; the paper's
# collection holds ~156 documents per video, the large bank is a stand-in for
# a shared knowledge base.
VIDEO_22S = RetrievalConfig("22 s video 220x336x336, 12 scenes, 156 docs", 220, 336, 336, 12,
                            156, 768, 3, 3, 0.6)
VIDEO_22S_BANK = RetrievalConfig("22 s video 220x336x336, 12 scenes, 100k docs", 220, 336, 336,
                                 12, 100_000, 768, 3, 3, 0.6)


def make_video(rc: RetrievalConfig, seed: int) -> np.ndarray:
    """uint8 frames [NF][H][W][3]: each scene is a random base image with its
    own colour range; every frame adds small noise and a slow brightness drift
    (so consecutive frames of a scene are similar, scene cuts are not)."""
    rng = host_rng(seed, "video")
    cuts = np.sort(rng.choice(np.arange(1, rc.n_frames), size=rc.n_scenes - 1, replace=False))
    scene_of = np.searchsorted(cuts, np.arange(rc.n_frames), side="right")
    bases = []
    for _ in range(rc.n_scenes):
        lo = rng.integers(0, 160, size=3)
        span = rng.integers(20, 96, size=3)
        bases.append(lo + rng.random((rc.height, rc.width, 3)) * span)
    out = np.empty((rc.n_frames, rc.height, rc.width, 3), dtype=np.uint8)
    for i in range(rc.n_frames):
        b = bases[scene_of[i]]
        noise = rng.normal(0.0, 2.0, size=b.shape)
        out[i] = np.clip(b + noise + 0.3 * (i % 7), 0, 255).astype(np.uint8)
    return out


def make_embeddings(n: int, dim: int, seed: int, name: str) -> np.ndarray:
    """float32 rows N(0, 1) (stand-ins for CLIP embeddings)."""
    return host_rng(seed, name).normal(size=(n, dim)).astype(np.float32)


def make_retrieval(rc: RetrievalConfig, seed: int):
    """(frames uint8 [NF][H][W][3], frame embeddings [NF][D], document
    embeddings [ND][D]); a few documents are planted near some frames so
    that retrieval has clear winners."""
    frames = make_video(rc, seed)
    femb = make_embeddings(rc.n_frames, rc.dim, seed, "frame_emb")
    demb = make_embeddings(rc.n_docs, rc.dim, seed, "doc_emb")
    rng = host_rng(seed, "planted_docs")
    for i in range(0, rc.n_frames, max(1, rc.n_frames // 8)):
        j = int(rng.integers(0, rc.n_docs))
        demb[j] = femb[i] + 0.5 * rng.normal(size=rc.dim).astype(np.float32)
    return frames, femb, demb
