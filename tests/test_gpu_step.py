"""The decode step as one launch (vbq_step_run) through the C ABI.

  * every y of a step equals, bit for bit, the y of the same GEMV launched on
    its own (same per-entry products, row sums and order), and matches the
    oracle within the 2e-3 rule and the float32 bound;
  * a genuinely dependent chain: GEMV i writes its y as fp16 and GEMV i+1
    reads that buffer as its x, so a missing wait would read stale inputs;
  * the 131M-class and 9B-class steps, a bucketed head written through a row
    map, repeated runs (bitwise identical), and the bounded wait: with a spin
    limit of one poll the launch still ends and reports the timeout in its
    status word, and the next normal run is correct.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import matmul as omatmul  # noqa: E402
from paper_2607_02893_amd import synth  # noqa: E402
from tests import parity  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def vbq():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02893_amd import vbq as v
    return v


def _say(msg):
    print(msg, flush=True)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _build(vbq, specs, seed):
    """Pack every matrix, draw its x, allocate its y; returns (mats, gemvs)."""
    mats, gemvs = [], []
    for spec in specs:
        bits, q, s = synth.make_matrix(spec, seed)
        x = synth.make_x(spec, seed)[0]
        blob, d = vbq.pack_codes(q, s, bits)
        Wp = vbq.PackedMatrix(blob, d)
        xd = _dev(x)
        y = torch.full((spec.N,), float("nan"), dtype=torch.float32, device="cuda")
        mats.append((spec, bits, q, s, x, Wp, xd, y))
        gemvs.append((d, Wp.blob.data_ptr(), xd.data_ptr(), y.data_ptr(), 0, 0))
    return mats, gemvs


def _check_step(vbq, specs, seed, what, oracle_every=1):
    mats, gemvs = _build(vbq, specs, seed)
    step = vbq.Step(gemvs)
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    worst = 0.0
    for i, (spec, bits, q, s, x, Wp, xd, y) in enumerate(mats):
        ys = y.cpu().numpy()
        ref = Wp.gemv(xd).cpu().numpy()
        assert np.array_equal(ys, ref), f"{what}: GEMV {i} ({spec.name} L{spec.layer}) differs from its own launch"
        if i % oracle_every == 0 or i == len(mats) - 1:
            ystar = omatmul.gemv(q, s, x)
            worst = max(worst, parity.check(ys, ystar, omatmul.row_magnitude(q, s, x), what=f"{what} {i}"))
            parity.check_bound(ys, ystar, parity.fp32_bound(q, s, bits, x), what=f"{what} {i}")
    # a second run gives the same bits
    ys0 = [m[7].clone() for m in mats]
    for m in mats:
        m[7].fill_(float("nan"))
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    for a, m in zip(ys0, mats):
        assert torch.equal(a, m[7])
    _say(f"{what}: {len(mats)} GEMVs in one launch, bitwise equal to per-GEMV launches; max rel err {worst:.2e}")


def test_step_131m_class(vbq):
    wl = synth.workload(1)
    _check_step(vbq, wl.matrices, wl.seed, "131M-class step")


def test_step_9b_class_layers_and_head(vbq):
    """Two 9B-class layers (Q|K|V, O, gate|up, down: two tiles per round and
    eight-unit tiles) and the 128256-row head (2004 tiles, eight rounds)."""
    wl = synth.workload(3)
    specs = [m for m in wl.matrices if m.layer in (0, 1)] + [wl.matrices[-1]]
    _check_step(vbq, specs, wl.seed, "9B-class layers 0-1 + head", oracle_every=3)


def test_step_dependent_chain(vbq):
    """y_i (fp16) is the x of GEMV i+1, so every GEMV needs its predecessor's
    whole output: the one-launch step equals the per-GEMV chain bit for bit."""
    dims = [1024, 2048, 512, 1024, 768]
    specs = [synth.MatrixSpec("c", i, 0, dims[i + 1], dims[i]) for i in range(len(dims) - 1)]
    packed = []
    for spec in specs:
        bits, q, s = synth.make_matrix(spec, 131)
        blob, d = vbq.pack_codes(q, s, bits)
        Wp = vbq.PackedMatrix(blob, d)
        packed.append((spec, Wp))
    # each layer grows the values by ~30x (the 8-bit groups): start small so the
    # whole chain stays inside fp16's normal range
    x0 = _dev(synth.make_x(specs[0], 131)[0] * np.float16(2.0 ** -14))
    bufs = [x0] + [torch.empty(sp.N, dtype=torch.float16, device="cuda") for sp in specs]
    gemvs = []
    for i, (spec, Wp) in enumerate(packed):
        d = Wp.call_desc(torch.float16)
        gemvs.append((d, Wp.blob.data_ptr(), bufs[i].data_ptr(), bufs[i + 1].data_ptr(), 0, 0))
    step = vbq.Step(gemvs)
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    got = [b.clone() for b in bufs[1:]]
    # the same chain, one launch per GEMV
    ref_bufs = [x0] + [torch.empty(sp.N, dtype=torch.float16, device="cuda") for sp in specs]
    for i, (spec, Wp) in enumerate(packed):
        Wp.gemv(ref_bufs[i], ref_bufs[i + 1])
    torch.cuda.synchronize()
    for i, (g, r) in enumerate(zip(got, ref_bufs[1:])):
        assert torch.isfinite(r.float()).all() and r.float().abs().max() > 1e-3, f"chain {i}: fp16 range"
        assert torch.equal(g, r), f"chain GEMV {i}"
    _say(f"dependent chain of {len(specs)} GEMVs: equal to the per-GEMV chain")


def test_step_bucketed_head_and_fp16_output(vbq):
    """Row buckets written through their row maps into one y, and an fp16 y."""
    spec = synth.MatrixSpec("h", 0, 4, 5000, 1024, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 137)
    x = synth.make_x(spec, 137)[0]
    xd = _dev(x)
    Wb = vbq.BucketedMatrix(vbq.pack_row_buckets(q, s, bits), spec.N, spec.K)
    y = torch.full((spec.N,), float("nan"), dtype=torch.float32, device="cuda")
    o_spec = synth.MatrixSpec("o", 1, 1, 768, 1024)
    ob, oq, os_ = synth.make_matrix(o_spec, 139)
    blob, d = vbq.pack_codes(oq, os_, ob)
    Wo = vbq.PackedMatrix(blob, d)
    y16 = torch.empty(768, dtype=torch.float16, device="cuda")
    gemvs = [(p.desc, p.blob.data_ptr(), xd.data_ptr(), y.data_ptr(), rows.data_ptr(), spec.N)
             for _, p, rows in Wb.parts]
    gemvs.append((Wo.call_desc(torch.float16), Wo.blob.data_ptr(), xd.data_ptr(), y16.data_ptr(), 0, 0))
    step = vbq.Step(gemvs)
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    assert torch.equal(y, Wb.gemv(xd))
    assert torch.equal(y16, Wo.gemv(xd, y_dtype=torch.float16))
    parity.check(y.cpu().numpy(), omatmul.gemv(q, s, x), omatmul.row_magnitude(q, s, x), what="bucketed head")


def test_step_bounded_wait_reports_a_timeout(vbq):
    """A spin limit of one poll: workgroups with no tile in the first GEMV reach
    the wait for it at once, give up, and the launch still ends with the
    status word set; a normal run afterwards is complete and correct."""
    wl = synth.workload(1)
    mats, gemvs = _build(vbq, wl.matrices[:6], wl.seed)
    step = vbq.Step(gemvs)
    assert step.run(spin_limit=1) == 0
    torch.cuda.synchronize()
    assert step.status() == 1
    assert step.run() == 0
    torch.cuda.synchronize()
    assert step.status() == 0
    for spec, bits, q, s, x, Wp, xd, y in mats:
        assert torch.equal(y, Wp.gemv(xd))
