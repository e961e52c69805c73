"""swan_decode_attention captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

A decode call enqueues only kernels (and, for a batch mixing k_pad on the GQA
or fp32 paths, event fork / join with the library's side streams), so a serving
loop can capture it.  Each
replay must give the eager call's output bit for bit (decode is deterministic),
with the program's own eager work and synchronisations between the replays, and
a replay after new queries are written into the captured input must match an
eager call on them.  The lengths and k are host arguments, fixed at capture.
"""
import sys

import numpy as np
import pytest

from tests.test_gpu_parity import _build

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("Hq,Hkv,ks,dtype", [(8, 8, [48, 48, 48], "f16"),
                                             (8, 8, [32, 48, 96], "f16"),  # fused launch
                                             (8, 2, [64, 64, 64], "f16"),  # GQA
                                             (8, 2, [32, 48, 96], "f16"),  # side streams
                                             (4, 4, [40, 64, 24], "f32")])
def test_decode_graph_replays_match_eager(gpu_device, swan_mod, torch_mod, Hq, Hkv, ks, dtype):
    torch = torch_mod
    _log(f"graph Hq={Hq} Hkv={Hkv} k={ks} {dtype}")
    Ls = [900, 333, 1]
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=3, Hq=Hq,
                                                Hkv=Hkv, L=Ls, b=16, k_active=ks, dtype=dtype)
    tdt = torch.float16 if dtype == "f16" else torch.float32
    gen = torch.Generator(device=gpu_device)
    gen.manual_seed(4242)
    q = torch.randn(3, Hq, 128, generator=gen, device=gpu_device).to(tdt)
    out_g = torch.empty_like(q)
    ref = cache.decode(q, tqk, tvo)  # eager; also sizes the workspace before capture
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cache.decode(q, tqk, tvo, out=out_g)
    for rep in range(4):
        g.replay()
        other = cache.decode(torch.flip(q, dims=[1]), tqk, tvo)  # eager work in between
        torch.cuda.synchronize()
        assert torch.equal(out_g, ref), f"replay {rep}"
        assert torch.isfinite(other).all()
    # new queries in the captured input
    q.copy_(torch.randn(3, Hq, 128, generator=gen, device=gpu_device).to(tdt))
    ref2 = cache.decode(q, tqk, tvo)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(out_g, ref2)
    assert not torch.equal(ref2, ref)
    del g
