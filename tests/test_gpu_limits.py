"""The launch shapes at their limits, against the oracle (pages and ring bit-exact,
outputs within 2e-3): the largest batch (64 sequences, ragged lengths, per-sequence k
spread over several k_pad groups), and the largest dense buffer (4096 tokens, which
the buffer wave stages in LDS), with sparse pages behind it and without."""
import sys

import numpy as np
import pytest

import swan_inputs as si
from tests import swan_cases as C
from tests.test_gpu_parity import _build, _decode_check

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_largest_batch(gpu_device, swan_mod, torch_mod):
    B = 64
    r = si.rng_for(1234)
    Ls = [int(x) for x in r.integers(1, 400, B)]
    ks = [int(x) for x in r.choice([8, 24, 32, 48, 64, 96, 128], B)]
    _log(f"B=64, L {min(Ls)}..{max(Ls)}, k from {sorted(set(ks))}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=4, Hkv=2,
                                                L=Ls, b=16, k_active=ks, dtype="f16",
                                                chunks=[150, 1, 300])
    for bi in range(B):
        C.compare_unit(cache, oc[bi][bi % 2], bi, bi % 2, Ls[bi], np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


@pytest.mark.parametrize("Hq,Hkv,Ls", [(4, 4, [5000, 3000]),    # MHA, pages behind the buffer
                                       (8, 2, [4200, 4096]),    # GQA
                                       (2, 2, [4096, 1])])      # all in the buffer
def test_largest_buffer(gpu_device, swan_mod, torch_mod, Hq, Hkv, Ls):
    b = 4096
    _log(f"b=4096 Hq={Hq} Hkv={Hkv} L={Ls}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=Hq,
                                                Hkv=Hkv, L=Ls, b=b, k_active=[48, 64],
                                                dtype="f16", chunks=[2500, 1, 2600])
    for bi in range(2):
        for h in range(Hkv):
            C.compare_unit(cache, oc[bi][h], bi, h, Ls[bi], np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")
