"""vsr_retrieve_static (no allocation: the library's static scratch) against
vsr_retrieve (caller's workspace) through the C ABI. Both run the same
kernels on the same inputs, so every output is compared bit for bit; the
second call is smaller than the first (the static scratch still holds the
first call's partial lists), the third takes the other scoring kernel
(D not a multiple of 16). Sizes beyond the static scratch are refused."""
import dataclasses
import sys

import numpy as np
import pytest

from paper_2601_01513_amd import workload as W

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _outputs(r):
    import torch
    torch.cuda.synchronize()
    n = int(r.n_keys.cpu()[0])
    ns = int(r.n_sel.cpu()[0])
    return (n, r.top_idx.cpu().numpy()[:n].copy(), r.top_sim.cpu().numpy()[:n].copy(), ns,
            r.sel_idx.cpu().numpy()[:ns].copy(), r.sel_sim.cpu().numpy()[:ns].copy())


def _same(a, b):
    assert a[0] == b[0] and a[3] == b[3]
    for x, y in zip(a, b):
        if isinstance(x, np.ndarray):
            assert x.dtype == y.dtype and np.array_equal(x.view(np.uint32), y.view(np.uint32))


def _case(rc, seed, dim=None):
    import torch
    from paper_2601_01513_amd.binding import Retriever
    dim = dim or rc.dim
    frames, femb, demb = W.make_retrieval(dataclasses.replace(rc, dim=dim), seed)
    _say(f"case: {rc.name}, D {dim}, seed {seed}")
    r = Retriever(rc.n_frames, rc.height, rc.width, rc.n_docs, dim, rc.k, rc.K)
    fr, fe, de = (torch.tensor(a, device="cuda") for a in (frames, femb, demb))
    r.keyframes(fr, rc.theta)
    r.retrieve(fe, de)
    ref = _outputs(r)
    for t in (r.top_idx, r.top_sim, r.sel_idx, r.sel_sim, r.n_sel):
        t.fill_(-7)
    r.retrieve_static(fe, de)
    got = _outputs(r)
    _say(f"  {ref[0]} keyframes, {ref[3]} documents selected")
    _same(ref, got)
    return ref


def test_static_scratch_matches_workspace_entry_point():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    big = _case(W.VIDEO_22S_BANK, 0)          # 220 frames, 100k documents x 768
    small = _case(W.VIDEO_SMALL, 1)           # 40 frames, 300 documents x 64
    odd = _case(W.VIDEO_SMALL, 2, dim=50)     # the per-document kernel
    assert big[0] > small[0] > 0 and odd[0] > 0


def test_static_scratch_refuses_sizes_beyond_it():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2601_01513_amd import binding as B
    lib = B.load_library()
    assert lib.vsr_retrieve_workspace_size(220, 1 << 24, 3) > B.VSR_RETRIEVE_STATIC_BYTES
    buf = torch.zeros(1 << 12, dtype=torch.float32, device="cuda")
    p = buf.data_ptr()
    rc = lib.vsr_retrieve_static(p, p, p, 220, p, 1 << 24, 768, 3, 3, p, p, p, p, p, None)
    assert rc == B.VSR_ERANGE
    assert b"scratch" in lib.vsr_last_error(None)
