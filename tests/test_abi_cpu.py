"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/vsr.h declares, sizes workspaces and rejects bad
arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2601_01513_amd import binding as B
from paper_2601_01513_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libvsr.so not built (python -m paper_2601_01513_amd.build)")
    return B.load_library()


def test_header_symbols_are_exported():
    lib = _lib()
    hdr = open(os.path.join(ROOT, "include", "vsr.h")).read()
    declared = set(re.findall(r"\b(vsr_[a-z_0-9]+)\s*\(", hdr))
    assert declared == set(B.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("cfg", W.CONFIGS, ids=lambda c: c.name)
def test_workspace_size_of_each_workload(cfg):
    _lib()
    n = B.workspace_size(B.make_config(cfg))
    assert n > 0 and n % 256 == 0
    # The prefix caches alone: 2 L Hkv P hd elements.
    e = 2 if cfg.dtype == W.BF16 else 4
    assert n > 2 * cfg.n_layers * cfg.n_kv_heads * cfg.n_prefix * cfg.head_dim * e


@pytest.mark.parametrize("field,value", [
    ("n_heads", 5), ("head_dim", 64), ("d_model", 100), ("dtype", 7), ("max_cands", 0),
    ("max_cands", B.VSR_MAX_CANDS + 1), ("vocab", 0), ("max_prefix", 0), ("d_ff", 96),
    ("split_layers", -1), ("split_layers", W.B1_5.n_layers + 1), ("gemm_weights", 3),
    ("gemm_weights", -1), ("max_new", -1), ("max_new", 4097), ("split_mlp_layers", -1),
    ("split_mlp_layers", 2)])
def test_invalid_configs_have_no_workspace(field, value):
    _lib()
    c = B.make_config(W.B1_5)
    setattr(c, field, value)
    assert B.workspace_size(c) == 0


def test_create_rejects_bad_arguments():
    lib = _lib()
    c = B.make_config(W.TINY_F32)
    need = lib.vsr_workspace_size(ctypes.byref(c))
    h = ctypes.c_void_p()
    assert lib.vsr_create(ctypes.byref(c), None, need, None, ctypes.byref(h)) == B.VSR_EINVAL
    assert b"workspace" in lib.vsr_last_error(None)
    assert lib.vsr_create(ctypes.byref(c), 0x1008, need, None, ctypes.byref(h)) == B.VSR_EINVAL
    assert lib.vsr_create(ctypes.byref(c), 0x10000, need - 1, None, ctypes.byref(h)) == B.VSR_ENOMEM
    assert lib.vsr_create(None, 0x10000, need, None, ctypes.byref(h)) == B.VSR_EINVAL
    assert lib.vsr_create(ctypes.byref(c), 0x10000, need, None, None) == B.VSR_EINVAL
    bad = B.make_config(W.TINY_F32)
    bad.n_kv_heads = 3
    assert lib.vsr_create(ctypes.byref(bad), 0x10000, need, None, ctypes.byref(h)) == B.VSR_EINVAL
    assert b"n_kv_heads" in lib.vsr_last_error(None)


def test_null_context_calls_fail_cleanly():
    lib = _lib()
    assert lib.vsr_load_weights(None, None) == B.VSR_EINVAL
    assert lib.vsr_prefill(None, None, 0, None, 1) == B.VSR_EINVAL
    lens = (ctypes.c_int32 * 1)(1)
    assert lib.vsr_score(None, None, lens, 1, 1, None, None, None) == B.VSR_EINVAL
    assert lib.vsr_verify(None, None, 0, None, 1, None, lens, 1, 1, None, None, None) == \
        B.VSR_EINVAL
    lib.vsr_destroy(None)


def test_workspace_holds_the_fused_rows():
    """bf16 contexts size their activation rows for vsr_verify (prefix rows +
    candidate rows in one pass): more candidate tokens, more workspace, even
    where the prefix is the larger of the two; fp32 contexts do not fuse."""
    _lib()
    base = B.make_config(W.B7)
    more = B.make_config(W.B7, max_cand_len=W.B7.cand_len + 64)
    assert B.workspace_size(more) > B.workspace_size(base)
    f32 = B.make_config(W.TINY_F32)
    f32_more = B.make_config(W.TINY_F32, max_prefix=W.TINY_F32.n_prefix + 64)
    assert B.workspace_size(f32_more) > B.workspace_size(f32)


def test_workspace_grows_with_the_maxima():
    _lib()
    a = B.workspace_size(B.make_config(W.B7))
    b = B.workspace_size(B.make_config(W.B7, max_prefix=2 * W.B7.n_prefix))
    c = B.workspace_size(B.make_config(W.B7, max_cands=2 * W.B7.n_cands))
    assert b > a and c > a


def test_precise_layers_add_their_buffers():
    """Precise layers need [hi | lo] activation rows and q/k/v remainder
    planes: the workspace grows with split_layers (and is exactly the fast
    size at 0); fp32 contexts ignore the field."""
    _lib()
    sizes = [B.workspace_size(B.make_config(W.B7, split_layers=s)) for s in (0, 1, 2, 28)]
    assert sizes[0] < sizes[1] < sizes[2] < sizes[3]
    f = [B.workspace_size(B.make_config(W.TINY_F32, split_layers=s)) for s in (0, 1)]
    assert f[0] == f[1]


def test_default_precise_layers_follow_depth():
    assert B.default_split_layers(0) == 0
    assert B.default_split_layers(1) == 1
    assert B.default_split_layers(28) == 1
    assert B.default_split_layers(64) == 2
    # The feed-forward block is split in the precise layers of deep models only.
    assert B.default_split_mlp_layers(28, 1) == 0
    assert B.default_split_mlp_layers(64, 2) == 2
    assert B.make_config(W.B7).split_mlp_layers == 0
    assert B.make_config(W.B32).split_mlp_layers == 2


def test_align_select_rejects_bad_arguments():
    lib = _lib()
    ok = dict(ent=0x10000, frames=0x20000, M=4, NF=8, D=16, rel=0x30000, delta=0.05,
              strategy=B.VSR_SELECT_TWO_STAGE, align=0x40000, choice=0x50000)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.vsr_align_select(a["ent"], a["frames"], a["M"], a["NF"], a["D"], a["rel"],
                                    a["delta"], a["strategy"], a["align"], a["choice"], None)
    for bad, word in ((dict(ent=None), b"NULL"), (dict(choice=None), b"NULL"),
                      (dict(M=0), b"M must"), (dict(M=B.VSR_MAX_CANDS + 1), b"M must"),
                      (dict(NF=0), b"NF"), (dict(D=0), b"D must"), (dict(D=4097), b"D must"),
                      (dict(delta=-0.1), b"delta"), (dict(delta=float("nan")), b"delta"),
                      (dict(delta=float("inf")), b"delta"), (dict(strategy=3), b"strategy"),
                      (dict(strategy=-1), b"strategy")):
        assert call(**bad) == B.VSR_EINVAL, bad
        assert word in lib.vsr_last_error(None), (bad, lib.vsr_last_error(None))


def test_reliability_without_context_fails_cleanly():
    lib = _lib()
    lens = (ctypes.c_int32 * 1)(1)
    assert lib.vsr_reliability(None, None, lens, 1, 1, 0, 1, 0.05, None, None, None) == \
        B.VSR_EINVAL


def test_draft_without_context_fails_cleanly():
    lib = _lib()
    lens = (ctypes.c_int32 * 1)(1)
    assert lib.vsr_draft(None, None, lens, 1, 1, 1, None) == B.VSR_EINVAL


def test_draft_cache_is_sized_by_max_new():
    """The draft cache holds L layers of keys and values for max_cands
    branches of max_cand_len + max_new positions (64-aligned) in the
    activation type; the rotary table gains max_new positions."""
    _lib()
    cfg = W.B1_5
    base = B.workspace_size(B.make_config(cfg, split_layers=0))
    for n in (1, 64, 4096):
        grown = B.workspace_size(B.make_config(cfg, split_layers=0, max_new=n))
        npos = -(-cfg.n_cands * (cfg.cand_len + n) // 64) * 64
        cache = 2 * cfg.n_layers * cfg.n_kv_heads * npos * cfg.head_dim * 2
        rope = n * cfg.head_dim * 4      # (cos, sin) float pairs of the extra positions
        # attention partials may grow too (a decode block walks every branch's
        # keys, so the key split may take more chunks), at most to 64 chunks
        T = cfg.n_cands * cfg.cand_len
        parts = 64 * T * cfg.n_heads * (cfg.head_dim * 4 + 8)
        extra = grown - base - cache - rope
        assert 0 <= extra <= parts + 4 * 256, (n, grown - base, cache + rope)


def test_fp32_contexts_take_no_gemm_weight_format():
    _lib()
    c = B.make_config(W.TINY_F32, gemm_weights=B.VSR_F16)
    assert B.workspace_size(c) == 0
    for g in (0, B.VSR_BF16, B.VSR_F16):
        assert B.workspace_size(B.make_config(W.B1_5, gemm_weights=g)) > 0


def test_weights_to_f16_rejects_bad_arguments():
    lib = _lib()
    assert lib.vsr_weights_to_f16(None, 0x1000, 8, None) == B.VSR_EINVAL
    assert lib.vsr_weights_to_f16(0x1008, 0x20000, 8, None) == B.VSR_EINVAL   # misaligned
    assert b"aligned" in lib.vsr_last_error(None)
    assert lib.vsr_weights_to_f16(0x10000, 0x10010, 64, None) == B.VSR_EINVAL  # overlap
    assert b"overlap" in lib.vsr_last_error(None)
    assert lib.vsr_weights_to_f16(None, None, 0, None) == B.VSR_OK             # nothing to do


def test_retrieval_calls_reject_bad_arguments():
    lib = _lib()
    ok = dict(frames=0x10000, NF=8, H=4, W=4, theta=0.5, hist=0x20000, inter=0x30000,
              key_idx=0x40000, n_keys=0x50000)

    def kf(**kw):
        a = dict(ok, **kw)
        return lib.vsr_keyframes(a["frames"], a["NF"], a["H"], a["W"], a["theta"], a["hist"],
                                 a["inter"], a["key_idx"], a["n_keys"], None)
    for bad in (dict(frames=None), dict(frames=0x10008), dict(NF=0), dict(NF=65537),
                dict(H=0), dict(W=5000, H=5000), dict(theta=float("nan")), dict(n_keys=None)):
        assert kf(**bad) == B.VSR_EINVAL, bad
    assert lib.vsr_retrieve_workspace_size(8, 100, 3) > 0
    for nf, nd, k in ((0, 100, 3), (8, 0, 3), (8, 100, 0), (8, 100, 17)):
        assert lib.vsr_retrieve_workspace_size(nf, nd, k) == 0
    ws = lib.vsr_retrieve_workspace_size(8, 100, 3)
    r = dict(fe=0x10000, ki=0x20000, nk=0x30000, NF=8, docs=0x40000, ND=100, D=64, k=3, K=3,
             ws=0x50000, wsb=ws, ti=0x60000, ts=0x70000, si=0x80000, ss=0x90000, ns=0xA0000)

    def rt(**kw):
        a = dict(r, **kw)
        return lib.vsr_retrieve(a["fe"], a["ki"], a["nk"], a["NF"], a["docs"], a["ND"], a["D"],
                                a["k"], a["K"], a["ws"], a["wsb"], a["ti"], a["ts"], a["si"],
                                a["ss"], a["ns"], None)
    for bad, word in ((dict(docs=None), b"NULL"), (dict(D=0), b"D must"), (dict(D=1025), b"D must"),
                      (dict(K=0), b"K must"), (dict(K=65), b"K must"), (dict(k=17), b"k must"),
                      (dict(ws=0x50004), b"aligned"), (dict(wsb=ws - 1), b"smaller")):
        assert rt(**bad) == B.VSR_EINVAL, bad
        assert word in lib.vsr_last_error(None), (bad, lib.vsr_last_error(None))


def test_retrieve_static_rejects_bad_arguments_and_oversize():
    """Argument and size checks of the no-allocation retrieval run before any
    HIP call (the pointers below are never dereferenced)."""
    lib = _lib()
    r = dict(fe=0x10000, ki=0x20000, nk=0x30000, NF=220, docs=0x40000, ND=100_000, D=768, k=3,
             K=3, ti=0x60000, ts=0x70000, si=0x80000, ss=0x90000, ns=0xA0000)

    def rs(**kw):
        a = dict(r, **kw)
        return lib.vsr_retrieve_static(a["fe"], a["ki"], a["nk"], a["NF"], a["docs"], a["ND"],
                                       a["D"], a["k"], a["K"], a["ti"], a["ts"], a["si"],
                                       a["ss"], a["ns"], None)
    for bad, word in ((dict(docs=None), b"NULL"), (dict(D=0), b"D must"), (dict(K=65), b"K must"),
                      (dict(k=17), b"k must"), (dict(docs=0x40004), b"aligned")):
        assert rs(**bad) == B.VSR_EINVAL, bad
        assert word in lib.vsr_last_error(None), (bad, lib.vsr_last_error(None))
    assert lib.vsr_retrieve_workspace_size(220, 1 << 24, 3) > B.VSR_RETRIEVE_STATIC_BYTES
    assert lib.vsr_retrieve_workspace_size(220, 1_000_000, 3) <= B.VSR_RETRIEVE_STATIC_BYTES
    assert rs(ND=1 << 24) == B.VSR_ERANGE
    assert b"scratch" in lib.vsr_last_error(None)


def test_set_checks_without_context_fails_cleanly():
    lib = _lib()
    assert lib.vsr_set_checks(None, B.VSR_CHECK_IDS) == B.VSR_EINVAL
    assert (B.VSR_EID, B.VSR_ENONFINITE) == (-6, -7)
