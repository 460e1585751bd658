"""ctypes binding of libvsr.so (C ABI: include/vsr.h).

Argument marshalling only: every step of the scoring pass runs inside the HIP
library. Torch tensors supply device memory and the stream. If the library is
not built, loading fails loudly; there is no other path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvsr.so")

VSR_OK, VSR_EINVAL, VSR_ESTATE, VSR_ERANGE, VSR_ENOMEM, VSR_EHIP = 0, -1, -2, -3, -4, -5
VSR_EID, VSR_ENONFINITE = -6, -7
VSR_CHECK_IDS, VSR_CHECK_FINITE = 1, 2
VSR_F32, VSR_BF16, VSR_F16 = 0, 1, 2
GEMM_WEIGHT_KEYS = ("wqkv", "wo", "wgu", "wdown")  # per layer, plus lm_head
VSR_MAX_CANDS = 256
VSR_RETRIEVE_STATIC_BYTES = 32 << 20

EXPORTS = ["vsr_workspace_size", "vsr_create", "vsr_load_weights", "vsr_prefill",
           "vsr_score", "vsr_verify", "vsr_reliability", "vsr_draft", "vsr_align_select", "vsr_weights_to_f16",
           "vsr_keyframes", "vsr_retrieve_workspace_size", "vsr_retrieve", "vsr_retrieve_static",
           "vsr_last_error",
           "vsr_destroy", "vsr_set_checks", "vsr_profile_enable", "vsr_profile_read"]

VSR_SELECT_TWO_STAGE, VSR_SELECT_ADDITION, VSR_SELECT_INVERT = 0, 1, 2
SELECT_STRATEGIES = {"two_stage": VSR_SELECT_TWO_STAGE, "addition": VSR_SELECT_ADDITION,
                     "invert": VSR_SELECT_INVERT}

VSR_STAGE_KINDS = 16
VSR_STAGES = 4 * VSR_STAGE_KINDS
VSR_PROFILE_ALL = (1 << VSR_STAGE_KINDS) - 1
STAGE_KINDS = ["embed", "rmsnorm", "qkv_rope", "attention", "attn_merge", "o_proj",
               "gate_up_swiglu", "down_proj", "lm_inputs", "lm_head_lse", "lse_gather",
               "sum_argmax", "row_tables", "copy", "tail_proj", "cand_attention"]
STAGE_NAMES = ([f"prefill.{k}" for k in STAGE_KINDS] + [f"score.{k}" for k in STAGE_KINDS]
               + [f"draft.{k}" for k in STAGE_KINDS] + [f"verify.{k}" for k in STAGE_KINDS])


class VsrConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("max_prefix", ctypes.c_int32), ("max_cands", ctypes.c_int32),
                ("max_cand_len", ctypes.c_int32), ("split_layers", ctypes.c_int32),
                ("gemm_weights", ctypes.c_int32), ("max_new", ctypes.c_int32),
                ("split_mlp_layers", ctypes.c_int32)]


_PP = ctypes.POINTER(ctypes.c_void_p)


class VsrWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("final_norm", ctypes.c_void_p), ("attn_norm", _PP), ("wqkv", _PP),
                ("wo", _PP), ("ffn_norm", _PP), ("wgu", _PP), ("wdown", _PP)]


class VsrError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"vsr error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libvsr.so (raises if it has not been built). The path defaults to
    the in-tree build; the VSR_LIBRARY environment variable names another
    build of the same library (e.g. to compare two builds on one machine)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("VSR_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2601_01513_amd.build`")
    lib = ctypes.CDLL(path)
    lib.vsr_workspace_size.argtypes = [ctypes.POINTER(VsrConfig)]
    lib.vsr_workspace_size.restype = ctypes.c_size_t
    lib.vsr_create.argtypes = [ctypes.POINTER(VsrConfig), ctypes.c_void_p, ctypes.c_size_t,
                               ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    lib.vsr_create.restype = ctypes.c_int
    lib.vsr_load_weights.argtypes = [ctypes.c_void_p, ctypes.POINTER(VsrWeights)]
    lib.vsr_load_weights.restype = ctypes.c_int
    lib.vsr_prefill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                ctypes.c_void_p, ctypes.c_int32]
    lib.vsr_prefill.restype = ctypes.c_int
    lib.vsr_score.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                              ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_int32,
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.vsr_score.restype = ctypes.c_int
    lib.vsr_verify.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                               ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                               ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_int32,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.vsr_verify.restype = ctypes.c_int
    lib.vsr_reliability.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p]
    lib.vsr_reliability.restype = ctypes.c_int
    lib.vsr_draft.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                              ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
    lib.vsr_draft.restype = ctypes.c_int
    lib.vsr_align_select.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_float, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p]
    lib.vsr_align_select.restype = ctypes.c_int
    lib.vsr_weights_to_f16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p]
    lib.vsr_weights_to_f16.restype = ctypes.c_int
    lib.vsr_keyframes.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p]
    lib.vsr_keyframes.restype = ctypes.c_int
    lib.vsr_retrieve_workspace_size.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
    lib.vsr_retrieve_workspace_size.restype = ctypes.c_size_t
    lib.vsr_retrieve.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                 ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                 ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p]
    lib.vsr_retrieve.restype = ctypes.c_int
    lib.vsr_retrieve_static.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.vsr_retrieve_static.restype = ctypes.c_int
    lib.vsr_last_error.argtypes = [ctypes.c_void_p]
    lib.vsr_last_error.restype = ctypes.c_char_p
    lib.vsr_destroy.argtypes = [ctypes.c_void_p]
    lib.vsr_destroy.restype = None
    lib.vsr_set_checks.argtypes = [ctypes.c_void_p, ctypes.c_int]
    lib.vsr_set_checks.restype = ctypes.c_int
    lib.vsr_profile_enable.argtypes = [ctypes.c_void_p, ctypes.c_int]
    lib.vsr_profile_enable.restype = ctypes.c_int
    lib.vsr_profile_read.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_int32)]
    lib.vsr_profile_read.restype = ctypes.c_int
    _lib = lib
    return lib


def default_split_layers(n_layers: int) -> int:
    """Precise leading layers for a decoder of this depth: one up to 63 layers,
    two at 64 (rounding amplification grows with depth)."""
    return min(n_layers, max(1, n_layers // 32))


def default_split_mlp_layers(n_layers: int, split_layers: int) -> int:
    """Precise layers whose feed-forward block is split too: all of them past
    32 layers, none up to 32 (measured against the oracle: 28 layers stay
    well inside the per-token bound with a plain FFN; 64 layers do not)."""
    return split_layers if n_layers > 32 else 0


def make_config(cfg, max_prefix: Optional[int] = None, max_cands: Optional[int] = None,
                max_cand_len: Optional[int] = None, split_layers: Optional[int] = None,
                gemm_weights: int = 0, max_new: int = 0,
                split_mlp_layers: Optional[int] = None) -> VsrConfig:
    """vsr_config from a workload.VerifierConfig (maxima default to its sizes;
    split_layers defaults to default_split_layers(n_layers), split_mlp_layers
    to default_split_mlp_layers; max_new = 0 reserves no draft cache)."""
    if split_layers is None:
        split_layers = default_split_layers(cfg.n_layers)
    if split_mlp_layers is None:
        split_mlp_layers = default_split_mlp_layers(cfg.n_layers, split_layers)
    return VsrConfig(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                     cfg.d_ff, cfg.vocab, cfg.rms_eps, cfg.rope_base, cfg.dtype,
                     max_prefix or cfg.n_prefix, max_cands or cfg.n_cands,
                     max_cand_len or cfg.cand_len, split_layers, gemm_weights, max_new,
                     split_mlp_layers)


def workspace_size(c: VsrConfig) -> int:
    return load_library().vsr_workspace_size(ctypes.byref(c))


def _ptr(t) -> int:
    return 0 if t is None else t.data_ptr()


class Verifier:
    """One vsr context: workspace, borrowed weights and the current prefix.

    gemm_weights (bf16 models): "f16" keeps fp16 copies of the GEMM weight
    matrices (the bf16 values, exact for magnitudes >= 2^-17), which the GEMMs
    load without conversion; "bf16" uses the given tensors as they are.
    max_new: the most tokens draft() may generate per branch (0: no drafting).
    """

    def __init__(self, cfg, weights: Dict, device="cuda", stream=None,
                 max_prefix=None, max_cands=None, max_cand_len=None, split_layers=None,
                 gemm_weights: str = "f16", max_new: int = 0, split_mlp_layers=None):
        import torch
        self._torch = torch
        self.lib = load_library()
        self.cfg = cfg
        if gemm_weights not in ("f16", "bf16"):
            raise ValueError("gemm_weights must be 'f16' or 'bf16'")
        self.gemm_f16 = cfg.dtype == VSR_BF16 and gemm_weights == "f16"
        self.c = make_config(cfg, max_prefix, max_cands, max_cand_len, split_layers,
                             VSR_F16 if self.gemm_f16 else 0, max_new, split_mlp_layers)
        size = self.lib.vsr_workspace_size(ctypes.byref(self.c))
        if size == 0:
            raise VsrError(VSR_EINVAL, "unsupported config")
        self.device = torch.device(device)
        self.workspace = torch.empty(size, dtype=torch.uint8, device=self.device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        h = ctypes.c_void_p()
        rc = self.lib.vsr_create(ctypes.byref(self.c), self.workspace.data_ptr(), size,
                                 self.stream.cuda_stream, ctypes.byref(h))
        if rc != VSR_OK:
            raise VsrError(rc, self.lib.vsr_last_error(None).decode())
        self.h = h
        self.load_weights(weights)

    def _check(self, rc: int):
        if rc != VSR_OK:
            raise VsrError(rc, self.lib.vsr_last_error(self.h).decode())

    def load_weights(self, w: Dict):
        if self.gemm_f16:  # one-time fp16 copies of the GEMM matrices
            f16 = lambda t: weights_to_f16(t, self.stream)  # noqa: E731
            w = dict(w, lm_head=f16(w["lm_head"]),
                     layers=[dict(lw, **{k: f16(lw[k]) for k in GEMM_WEIGHT_KEYS})
                             for lw in w["layers"]])
        self.weights = w  # keep the borrowed tensors alive
        L = len(w["layers"])
        arrs = {}
        for k in ("attn_norm", "wqkv", "wo", "ffn_norm", "wgu", "wdown"):
            arrs[k] = (ctypes.c_void_p * max(L, 1))(*[_ptr(lw[k]) for lw in w["layers"]])
        self._arrs = arrs
        cw = VsrWeights(_ptr(w["embed"]), _ptr(w["lm_head"]), _ptr(w["final_norm"]),
                        *[ctypes.cast(arrs[k], _PP) for k in
                          ("attn_norm", "wqkv", "wo", "ffn_norm", "wgu", "wdown")])
        self._check(self.lib.vsr_load_weights(self.h, ctypes.byref(cw)))

    def prefill(self, visual, ids):
        """visual: device [Pv][d] (config dtype) or None; ids: device int32 [Pt] or None."""
        nv = 0 if visual is None else int(visual.shape[0])
        nt = 0 if ids is None else int(ids.shape[0])
        self._keep = (visual, ids)
        self._check(self.lib.vsr_prefill(self.h, _ptr(visual), nv, _ptr(ids), nt))

    def score(self, cand_ids, cand_len: Sequence[int], out=None):
        """cand_ids: device int32 [M][Cmax]; cand_len: host ints [M].

        Returns device tensors (logprobs [M][Cmax] f32, scores [M] f32,
        argmax [1] int32), valid once the stream is synchronised.
        """
        torch = self._torch
        M, cmax = int(cand_ids.shape[0]), int(cand_ids.shape[1])
        lens = (ctypes.c_int32 * M)(*[int(x) for x in cand_len])
        if out is None:
            out = (torch.empty((M, cmax), dtype=torch.float32, device=self.device),
                   torch.empty(M, dtype=torch.float32, device=self.device),
                   torch.empty(1, dtype=torch.int32, device=self.device))
        lp, sc, am = out
        self._check(self.lib.vsr_score(self.h, _ptr(cand_ids), lens, M, cmax, _ptr(lp),
                                       _ptr(sc), _ptr(am)))
        return lp, sc, am

    def verify(self, visual, ids, cand_ids, cand_len: Sequence[int], out=None):
        """prefill(visual, ids) and score(cand_ids, cand_len) as one fused
        pass; same arguments and outputs, and the prefix stays current."""
        torch = self._torch
        nv = 0 if visual is None else int(visual.shape[0])
        nt = 0 if ids is None else int(ids.shape[0])
        self._keep = (visual, ids)
        M, cmax = int(cand_ids.shape[0]), int(cand_ids.shape[1])
        lens = (ctypes.c_int32 * M)(*[int(x) for x in cand_len])
        if out is None:
            out = (torch.empty((M, cmax), dtype=torch.float32, device=self.device),
                   torch.empty(M, dtype=torch.float32, device=self.device),
                   torch.empty(1, dtype=torch.int32, device=self.device))
        lp, sc, am = out
        self._check(self.lib.vsr_verify(self.h, _ptr(visual), nv, _ptr(ids), nt, _ptr(cand_ids),
                                        lens, M, cmax, _ptr(lp), _ptr(sc), _ptr(am)))
        return lp, sc, am

    def reliability(self, branch_ids, branch_len: Sequence[int], yes_id: int, no_id: int,
                    delta: float, out=None):
        """Stage 1 of the two-stage verification against the current prefix.

        branch_ids: device int32 [M][Cmax]; branch_len: host ints [M], each >= 1.
        Returns device tensors (lp_yes_no [M][2] f32, rel [M] f32, keep [M]
        int32), valid once the stream is synchronised.
        """
        torch = self._torch
        M, cmax = int(branch_ids.shape[0]), int(branch_ids.shape[1])
        lens = (ctypes.c_int32 * M)(*[int(x) for x in branch_len])
        if out is None:
            out = (torch.empty((M, 2), dtype=torch.float32, device=self.device),
                   torch.empty(M, dtype=torch.float32, device=self.device),
                   torch.empty(M, dtype=torch.int32, device=self.device))
        lp, rel, keep = out
        self._check(self.lib.vsr_reliability(self.h, _ptr(branch_ids), lens, M, cmax,
                                             int(yes_id), int(no_id), float(delta), _ptr(lp),
                                             _ptr(rel), _ptr(keep)))
        return lp, rel, keep

    def draft(self, prompt_ids, prompt_len: Sequence[int], n_new: int, out=None):
        """Greedy parallel drafts (Eq. 5, 8-10) after the current prefix.

        prompt_ids: device int32 [M][Cmax]; prompt_len: host ints [M], each >= 1.
        Returns a device int32 tensor [M][n_new] of generated token ids, valid
        once the stream is synchronised.
        """
        torch = self._torch
        M, cmax = int(prompt_ids.shape[0]), int(prompt_ids.shape[1])
        lens = (ctypes.c_int32 * M)(*[int(x) for x in prompt_len])
        if out is None:
            out = torch.empty((M, int(n_new)), dtype=torch.int32, device=self.device)
        self._check(self.lib.vsr_draft(self.h, _ptr(prompt_ids), lens, M, cmax, int(n_new),
                                       _ptr(out)))
        return out

    def set_checks(self, ids: bool = True, finite: bool = True):
        """Call validator (vsr_set_checks): later calls wait for their stream
        and raise VsrError with code VSR_EID / VSR_ENONFINITE on a bad id or a
        non-finite result (their outputs are still written)."""
        self._check(self.lib.vsr_set_checks(
            self.h, (VSR_CHECK_IDS if ids else 0) | (VSR_CHECK_FINITE if finite else 0)))

    def profile(self, enable, kinds=None):
        """Turns per-stage kernel timing on or off (clears recorded launches).
        `kinds`: stage-kind names (STAGE_KINDS) to time; default all."""
        mask = 0
        if enable:
            mask = VSR_PROFILE_ALL if kinds is None else sum(1 << STAGE_KINDS.index(k) for k in kinds)
        self._check(self.lib.vsr_profile_enable(self.h, mask))

    def profile_read(self) -> Dict[str, tuple]:
        """{stage name: (summed ms, launches)} since the last read."""
        ms = (ctypes.c_double * VSR_STAGES)()
        n = (ctypes.c_int32 * VSR_STAGES)()
        self._check(self.lib.vsr_profile_read(self.h, ms, n))
        return {STAGE_NAMES[i]: (ms[i], n[i]) for i in range(VSR_STAGES) if n[i]}

    def close(self):
        if getattr(self, "h", None):
            self.lib.vsr_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def weights_to_f16(t, stream=None):
    """fp16 copy of a contiguous bf16 device tensor, rounded as the GEMMs
    round bf16 weights (vsr_weights_to_f16)."""
    import torch
    if t.dtype != torch.bfloat16 or not t.is_contiguous():
        raise VsrError(VSR_EINVAL, "weights_to_f16: contiguous bfloat16 tensor expected")
    lib = load_library()
    out = torch.empty(t.shape, dtype=torch.float16, device=t.device)
    st = stream if stream is not None else torch.cuda.current_stream(t.device)
    rc = lib.vsr_weights_to_f16(_ptr(t), _ptr(out), t.numel(), st.cuda_stream)
    if rc != VSR_OK:
        raise VsrError(rc, lib.vsr_last_error(None).decode())
    return out


def align_select(ent, frames, rel, delta: float, strategy: str = "two_stage", out=None,
                 stream=None):
    """Entity alignment (Eq. 14-15) and the final choice (Algorithm 1 or a
    Table 3 strategy). ent: device f32 [M][D]; frames: device f32 [NF][D];
    rel: device f32 [M]. Returns device tensors (align [M] f32, choice [1]
    int32), valid once the stream is synchronised."""
    import torch
    lib = load_library()
    M, D = int(ent.shape[0]), int(ent.shape[1])
    NF = int(frames.shape[0])
    if int(frames.shape[1]) != D or int(rel.shape[0]) != M:
        raise VsrError(VSR_EINVAL, "align_select: shapes of ent, frames and rel disagree")
    for t in (ent, frames, rel):
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise VsrError(VSR_EINVAL, "align_select: contiguous float32 tensors expected")
    if out is None:
        out = (torch.empty(M, dtype=torch.float32, device=ent.device),
               torch.empty(1, dtype=torch.int32, device=ent.device))
    align, choice = out
    st = stream if stream is not None else torch.cuda.current_stream(ent.device)
    rc = lib.vsr_align_select(_ptr(ent), _ptr(frames), M, NF, D, _ptr(rel), float(delta),
                              SELECT_STRATEGIES[strategy], _ptr(align), _ptr(choice),
                              st.cuda_stream)
    if rc != VSR_OK:
        raise VsrError(rc, lib.vsr_last_error(None).decode())
    return align, choice


class Retriever:
    """The retrieval stage on the device: keyframes (Eq. 1), then per-keyframe
    top-k documents and T* (Eq. 2-3). Holds the output and workspace tensors
    for one video size and document bank."""

    def __init__(self, n_frames: int, height: int, width: int, n_docs: int, dim: int, k: int,
                 K: int, device="cuda", stream=None):
        import torch
        self._torch = torch
        self.lib = load_library()
        self.NF, self.H, self.W, self.ND, self.D, self.k, self.K = (
            n_frames, height, width, n_docs, dim, k, K)
        dev = torch.device(device)
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.hist = torch.empty((n_frames, 3, 64), **i32)
        self.inter = torch.empty(n_frames, **i32)
        self.key_idx = torch.empty(n_frames, **i32)
        self.n_keys = torch.empty(1, **i32)
        size = self.lib.vsr_retrieve_workspace_size(n_frames, n_docs, k)
        if size == 0:
            raise VsrError(VSR_EINVAL, "unsupported retrieval sizes")
        self.ws = torch.empty(size, dtype=torch.uint8, device=dev)
        self.top_idx = torch.empty((n_frames, k), **i32)
        self.top_sim = torch.empty((n_frames, k), **f32)
        self.sel_idx = torch.empty(K, **i32)
        self.sel_sim = torch.empty(K, **f32)
        self.n_sel = torch.empty(1, **i32)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)

    def _check(self, rc):
        if rc != VSR_OK:
            raise VsrError(rc, self.lib.vsr_last_error(None).decode())

    def keyframes(self, frames, theta: float):
        """frames: device uint8 [NF][H][W][3] -> (key_idx, n_keys) device tensors."""
        self._frames = frames
        self._check(self.lib.vsr_keyframes(_ptr(frames), self.NF, self.H, self.W, float(theta),
                                           _ptr(self.hist), _ptr(self.inter),
                                           _ptr(self.key_idx), _ptr(self.n_keys),
                                           self.stream.cuda_stream))
        return self.key_idx, self.n_keys

    def retrieve(self, frame_emb, docs):
        """frame_emb: device f32 [NF][D]; docs: device f32 [ND][D]. Uses the
        keyframes of the last keyframes() call. Returns device tensors
        (top_idx [NF][k], top_sim, sel_idx [K], sel_sim, n_sel)."""
        self._emb = (frame_emb, docs)
        self._check(self.lib.vsr_retrieve(
            _ptr(frame_emb), _ptr(self.key_idx), _ptr(self.n_keys), self.NF, _ptr(docs),
            self.ND, self.D, self.k, self.K, _ptr(self.ws), self.ws.numel(), _ptr(self.top_idx),
            _ptr(self.top_sim), _ptr(self.sel_idx), _ptr(self.sel_sim), _ptr(self.n_sel),
            self.stream.cuda_stream))
        return self.top_idx, self.top_sim, self.sel_idx, self.sel_sim, self.n_sel

    def retrieve_static(self, frame_emb, docs):
        """retrieve() through vsr_retrieve_static: the library's static
        scratch instead of this object's workspace (no allocation in the call)."""
        self._emb = (frame_emb, docs)
        self._check(self.lib.vsr_retrieve_static(
            _ptr(frame_emb), _ptr(self.key_idx), _ptr(self.n_keys), self.NF, _ptr(docs),
            self.ND, self.D, self.k, self.K, _ptr(self.top_idx), _ptr(self.top_sim),
            _ptr(self.sel_idx), _ptr(self.sel_sim), _ptr(self.n_sel), self.stream.cuda_stream))
        return self.top_idx, self.top_sim, self.sel_idx, self.sel_sim, self.n_sel


def verifier_from_workload(wl, device="cuda", **kw) -> Verifier:
    return Verifier(wl.cfg, wl.weights, device=device, **kw)
