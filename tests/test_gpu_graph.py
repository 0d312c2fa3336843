"""HIP-graph capture of the library's calls (marked gpu).

The forward, the backward (workspace and no-allocation variants) and the
merge are captured once into a HIP graph and replayed several times, with
eager library work between the replays; every replay must reproduce the eager
results bit for bit.  Two layers: a small per-wave-kernel layer and one large
enough for the wide grid kernel (packed INT4 with a zero offset and the scale
gradient, so every output of the backward is covered).  The library issues no
memset, copy or synchronisation, so a caller may capture any of its calls."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2406_06385_amd import inputs as I

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def lr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_06385_amd import lrqat
    lrqat.load_library()
    return lrqat


def _bf16(a):
    return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()


def _same(a, b):
    return all(torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y) for x, y in zip(a, b))


CASES = [
    # m, k, T, r, bits, fmt, asymmetric
    (320, 264, 96, 16, 4, "q8", False),
    (2048, 4096, 256, 32, 4, "int_packed2", True),
]


@pytest.mark.parametrize("case", CASES, ids=[f"m{c[0]}k{c[1]}r{c[3]}{c[5]}{'z' if c[6] else ''}" for c in CASES])
def test_graph_replays_match_eager(lr, case):
    m, k, T, r, bits, fmt, asym = case
    _log(f"[graph {case}]")
    spec = lr.LayerSpec(m, k, r, float(r), bits, fmt, 0, 0, "bf16")
    W0 = torch.from_numpy(I.gen_w0(m, k, 91, 92, 0.02, 0.0)).cuda()
    A = torch.from_numpy(I.gen_a(m, r, k, 93)).cuda()
    B = torch.from_numpy(I.gen_b(r, k, 94, 0.05)).cuda()
    X = _bf16(I.gen_act(T, k, 95, 1.0, "bf16"))
    dY = _bf16(I.gen_act(T, m, 96, 1e-2, "bf16"))
    if asym:
        s, z, phi = lr.lrqat_init_from_weights(spec, W0, asymmetric=True)
    else:
        (s, phi), z = lr.lrqat_init_from_weights(spec, W0), None
    Y = torch.empty((T, m), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty((T, k), dtype=torch.bfloat16, device="cuda")
    dA = torch.empty((m, r), device="cuda")
    dB = torch.empty((r, k), device="cuda")
    ds = torch.empty(s.shape, device="cuda")
    dX2, dA2, dB2 = torch.empty_like(dX), torch.empty_like(dA), torch.empty_like(dB)
    W = torch.empty((m, k // 2), dtype=torch.uint8, device="cuda")
    wf = lr.workspace(lr.lrqat_forward_workspace_size(spec, T))
    wb = lr.workspace(lr.lrqat_backward_workspace_size(spec, T))

    def step():
        lr.lrqat_forward(spec, X, phi, s, A, B, Y=Y, ws=wf, z=z)
        lr.lrqat_backward(spec, X, phi, s, A, B, dY, dX=dX, dA=dA, dB=dB, ws=wb, z=z, ds=ds)
        lr.lrqat_backward_static(spec, X, phi, s, A, B, dY, dX=dX2, dA=dA2, dB=dB2, z=z)
        lr.lrqat_merge_to_int4(spec, phi, A, B, out=W)

    outs = (Y, dX, dA, dB, ds, dX2, dA2, dB2, W)
    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    assert _same([dX2, dA2, dB2], [ref[1], ref[2], ref[3]]), "the no-allocation backward differs from the backward"

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for t in outs:
            t.fill_(0) if t.dtype == torch.uint8 else t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert _same(outs, ref), f"replay {rep} differs from the eager step"
        step()  # eager work between replays
        torch.cuda.synchronize()
        assert _same(outs, ref)
