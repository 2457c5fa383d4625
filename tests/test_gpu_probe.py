"""The integer VALU throughput probe (a diagnostic beside the search): its
words equal the same chains computed on the host, so the measured ceiling
comes from the arithmetic it claims to run."""
import sys

import numpy as np
import pytest

import paper_2607_22242_amd as S

pytestmark = pytest.mark.gpu


def host_probe(blocks: int, iters: int, seed: int = 0x5EED) -> np.ndarray:
    m = np.uint64(0xFFFFFFFF)
    g = np.arange(blocks * 256, dtype=np.uint64)
    s = np.uint64(seed)
    x = (s ^ g) & m
    y = (s * np.uint64(3) + g) & m
    z = (s + (g << np.uint64(3))) & m
    w = (g * np.uint64(0x9E3779B9)) & m
    a = [(g + np.uint64(j * 0x01234567)) & m for j in range(8)]
    for _ in range(iters):
        for j in range(8):
            v = (a[j] + x) & m
            v = np.maximum(v, y)
            a[j] = np.where(v > z, v, w)
    r = np.zeros_like(g)
    for j in range(8):
        r ^= a[j]
    return r.astype(np.uint32)


@pytest.mark.parametrize("blocks,iters", [(1, 1), (3, 17), (2, 64)])
def test_probe_words_match_host(blocks, iters):
    import torch
    assert torch.cuda.is_available()
    print(f"probe blocks={blocks} iters={iters}", flush=True)
    sys.stdout.flush()
    out = torch.zeros(blocks * 256, dtype=torch.int32, device="cuda")
    ops = S.sched_valu_probe(blocks, iters, out)
    assert ops == blocks * 256 * iters * 32
    got = out.cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(got, host_probe(blocks, iters))
