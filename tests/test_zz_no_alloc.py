"""The allocation-free routing entry point (moe_route_permute_noalloc) against the workspace form
(moe_route_permute), through the C ABI: two calls in a row on the library's shared device scratch,
the second with a smaller input, every output bit-exact."""
import sys

import pytest
import torch

from paper_2606_26453_amd import moe
from tests.gpu_util import gpu_available, poison_

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda:0"


def _inputs(T, d, E, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    logits = torch.randn((T, E), generator=g, device=DEV)
    logits[::7, 1] = logits[::7, 0]      # exact ties: the lower id must win on both sides
    x = torch.randn((T, d), generator=g, device=DEV).to(torch.bfloat16)
    return logits, x


def _run(fn, logits, x, k, **kw):
    T, E = logits.shape
    R = T * k
    out = {"topk_idx": poison_(torch.empty((T, k), dtype=torch.int32, device=DEV)),
           "topk_w": poison_(torch.empty((T, k), dtype=torch.float32, device=DEV)),
           "offsets": poison_(torch.empty(E + 1, dtype=torch.int32, device=DEV)),
           "row_of_slot": poison_(torch.empty(R, dtype=torch.int32, device=DEV)),
           "token_of_row": poison_(torch.empty(R, dtype=torch.int32, device=DEV)),
           "x_perm": poison_(torch.empty((R, x.shape[1]), dtype=torch.bfloat16, device=DEV))}
    return fn(logits, x, k, **out, **kw)


@pytest.mark.parametrize("case", [((8192, 256, 64, 6), (1000, 128, 64, 6)),    # fine-grained, then smaller
                                  ((16384, 128, 8, 2), (300, 64, 8, 2)),        # Mixtral-like routing
                                  ((5000, 64, 256, 8), (17, 64, 256, 8))])      # E = 256
def test_noalloc_matches_workspace_form(case):
    print("no-alloc routing", case, flush=True)
    sys.stdout.flush()
    for i, (T, d, E, k) in enumerate(case):
        logits, x = _inputs(T, d, E, seed=40 + i)
        ref = _run(moe.moe_route_permute, logits, x, k)
        got = _run(moe.moe_route_permute_noalloc, logits, x, k)
        torch.cuda.synchronize()
        for name in ref:
            a, b = ref[name], got[name]
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            elif a.dtype == torch.float32:
                a, b = a.view(torch.int32), b.view(torch.int32)
            assert torch.equal(a, b), f"{name} differs (T={T}, E={E}, k={k})"


def test_noalloc_rejects_oversized():
    L = moe.lib()
    cap = L.moe_route_permute_noalloc_max_scratch_bytes()
    assert cap > 0
    # sizes whose histogram exceeds the scratch are refused on the host, before any launch
    T, E, k = 1 << 24, 256, 8
    assert L.moe_route_permute_workspace_bytes(T, E, k) > cap
    fake = 1 << 20
    st = L.moe_route_permute_noalloc(fake, None, T, 0, E, k, 1, fake, fake, fake, fake, fake, None, None)
    assert st == 2   # MOE_ERROR_NOT_SUPPORTED
    assert b"scratch" in L.moe_last_error()
