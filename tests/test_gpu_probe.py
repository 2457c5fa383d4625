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


def test_wave_or_matches_host():
    """The wave-wide OR through LDS (the search's skipping masks) equals the
    OR over each wave's active lanes, for 64-bit words whose low half often has
    bit 31 set (the high half must come back as it is, not filled with
    ones) and for the 32-bit form; lanes outside the branch write all ones.
    Waves with no active lane, one active lane and all lanes active are
    included."""
    import torch
    assert torch.cuda.is_available()
    blocks = 4
    n = blocks * 256
    print(f"wave-or probe blocks={blocks}", flush=True)
    rng = np.random.default_rng(2031)
    lo = rng.integers(0, 1 << 32, n, dtype=np.uint64)
    lo[rng.random(n) < 0.5] |= np.uint64(1 << 31)
    hi = rng.integers(0, 1 << 32, n, dtype=np.uint64) & np.uint64(0x0F0F00F0)
    x = (hi << np.uint64(32)) | lo
    active = (rng.random(n) < 0.6).astype(np.uint8)
    active[0:64] = 0           # a wave with no active lane
    active[64:128] = 0
    active[64 + 37] = 1        # a wave with one active lane
    active[128:192] = 1        # a wave with every lane active
    d_in = torch.from_numpy(x.view(np.int64)).cuda()
    d_act = torch.from_numpy(active).cuda()
    d_o64 = torch.zeros(n, dtype=torch.int64, device="cuda")
    d_o32 = torch.zeros(n, dtype=torch.int32, device="cuda")
    S.sched_wave_or_probe(d_in, d_act, blocks, d_o64, d_o32)
    o64 = d_o64.cpu().numpy().view(np.uint64)
    o32 = d_o32.cpu().numpy().view(np.uint32)
    want64 = np.full(n, np.uint64(0xFFFFFFFFFFFFFFFF), dtype=np.uint64)
    want32 = np.full(n, np.uint32(0xFFFFFFFF), dtype=np.uint32)
    for w in range(n // 64):
        sl = slice(64 * w, 64 * w + 64)
        on = active[sl] != 0
        if not on.any():
            continue
        r = np.bitwise_or.reduce(x[sl][on])
        r32 = np.bitwise_or.reduce(((x[sl][on] >> np.uint64(16)) & np.uint64(0xFFFFFFFF)))
        want64[sl][on] = r
        want32[sl][on] = np.uint32(r32)
    np.testing.assert_array_equal(o64, want64)
    np.testing.assert_array_equal(o32, want32)
