"""albireo_sample_noalloc (the entry point that allocates nothing) against albireo_sample: the same
kernels, so the outputs must be identical, on two calls in a row (the second on a smaller batch, so
that it runs on the scratch array the first one left behind)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01927_amd as alb

    return alb


def _both(alb, w):
    from workloads.device import to_device

    logits, u, p = to_device(w)
    ref = alb.sample(logits, u, p, n_top=w.n_top, V=w.V)
    got = alb.sample_noalloc(logits, u, p, n_top=w.n_top, V=w.V)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in ref], [t.cpu().numpy() for t in got]


def test_noalloc_matches_sample_twice(lib):
    for cfg, B, V, H in ((5, 64, 60013, 512), (3, 16, 20011, 300)):
        w = workloads.generate(cfg, B=B, V=V, H=H)
        _say("noalloc", cfg, B, V)
        ref, got = _both(lib, w)
        for name, r, g in zip(("ids", "logprobs", "top_ids", "top_logprobs", "flags"), ref, got):
            assert np.array_equal(r, g, equal_nan=True), "%s differs (cfg %d, B %d)" % (name, cfg, B)


def test_noalloc_rejects_shapes_over_the_scratch(lib):
    from paper_2606_01927_amd import AlbireoError, E_SCRATCH

    # 8192 rows of a V = 256000 bf16 vocabulary need 8192 * 7 chunks: far above the 32 MiB scratch
    B, V = 8192, 256000
    logits = torch.empty((1, V), dtype=torch.bfloat16, device="cuda").expand(B, V)
    u = torch.zeros(B, dtype=torch.float32, device="cuda")
    with pytest.raises(AlbireoError) as e:
        lib.sample_noalloc(logits, u, V=V)
    assert e.value.status == E_SCRATCH
