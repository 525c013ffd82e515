"""The no-allocation index build (moe_build_index_noalloc) against
moe_build_index through the C ABI: bit-exact outputs on two calls in a row,
the second with a smaller input (the static scratch keeps the first call's
contents, and nothing of it may leak into the second)."""
import numpy as np
import pytest
import torch

from paper_2601_05296_amd import binding as B
from paper_2601_05296_amd import synth

pytestmark = pytest.mark.gpu


def _outputs(T, E, k):
    i32 = dict(dtype=torch.int32, device="cuda")
    return [torch.full((E,), -7, **i32), torch.full((E + 1,), -7, **i32),
            torch.full((T * k,), -7, **i32), torch.full((T, k), -7, **i32),
            torch.full((T * k,), -7, **i32)]


@pytest.mark.parametrize("pattern", ["uniform", "skewed"])
def test_build_index_noalloc_matches_workspace_call(pattern):
    for T, E, k, seed in ((60000, 256, 8, 11), (3001, 64, 6, 12)):
        print("no-alloc index build: T=%d E=%d k=%d %s" % (T, E, k, pattern), flush=True)
        pop = None if pattern == "uniform" else 1.0 / np.arange(1, E + 1) ** 1.2
        ids = torch.from_numpy(synth.random_ids(T, E, k, seed=seed, popularity=pop)).cuda()
        ref = _outputs(T, E, k)
        wsb = B.moe_build_index_workspace_size(T, E, k)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_build_index(ids, T, E, k, *ref, ws, wsb)
        got = _outputs(T, E, k)
        B.moe_build_index_noalloc(ids, T, E, k, *got)
        torch.cuda.synchronize()
        for name, a, b in zip(("counts", "offsets", "eti", "tim", "slot_src"), got, ref):
            assert torch.equal(a, b), (name, T, E, k)
