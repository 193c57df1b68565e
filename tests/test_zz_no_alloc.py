"""vbq_step_run_noalloc (no workspace argument, the library's own scratch)
against vbq_step_run (a caller workspace) through the C ABI: two calls in a
row, the second on a smaller step, each bitwise equal to the workspace path,
with its status word written to the caller's word; a step beyond the
scratch's limit is refused before anything is launched."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2607_02893_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def vbq():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02893_amd import vbq as v
    return v


def _step(vbq, specs, seed):
    mats, gemvs = [], []
    for spec in specs:
        bits, q, s = synth.make_matrix(spec, seed)
        blob, d = vbq.pack_codes(q, s, bits)
        Wp = vbq.PackedMatrix(blob, d)
        xd = torch.from_numpy(np.ascontiguousarray(synth.make_x(spec, seed)[0])).cuda()
        y = torch.empty(spec.N, dtype=torch.float32, device="cuda")
        mats.append((Wp, xd, y))
        gemvs.append((d, Wp.blob.data_ptr(), xd.data_ptr(), y.data_ptr(), 0, 0))
    return vbq.Step(gemvs), mats


def _run_both(vbq, step, mats, status):
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    want = [m[2].clone() for m in mats]
    for m in mats:
        m[2].fill_(float("nan"))
    status.fill_(-1)
    assert step.run_noalloc(status) == 0
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for w, m in zip(want, mats):
        assert torch.equal(w, m[2])
    # each y is also what the GEMV launched on its own gives
    for Wp, xd, y in mats:
        assert torch.equal(y, Wp.gemv(xd))


def test_noalloc_step_matches_the_workspace_path(vbq):
    wl = synth.workload(1)
    status = torch.empty(1, dtype=torch.int32, device="cuda")
    big, big_mats = _step(vbq, wl.matrices, wl.seed)            # 49 GEMVs
    small, small_mats = _step(vbq, wl.matrices[5:12], wl.seed + 1)  # then 7 GEMVs
    _run_both(vbq, big, big_mats, status)
    _run_both(vbq, small, small_mats, status)
    assert small.run_noalloc(None) == 0                          # no status word wanted
    torch.cuda.synchronize()
    for Wp, xd, y in small_mats:
        assert torch.equal(y, Wp.gemv(xd))


def test_noalloc_step_refuses_more_gemvs_than_its_scratch_holds(vbq):
    lib = vbq.lib()
    A = 1 << 20  # never dereferenced: refused before any launch
    import ctypes
    assert lib.vbq_step_run_noalloc(ctypes.c_void_p(A), 513, 0, None, None) == 2
    assert lib.vbq_step_run_noalloc(ctypes.c_void_p(A), 0, 0, None, None) == 2
    assert lib.vbq_step_run_noalloc(None, 4, 0, None, None) == 1
    assert lib.vbq_step_run_noalloc(ctypes.c_void_p(A), 4, 0, ctypes.c_void_p(A + 2), None) == 7
