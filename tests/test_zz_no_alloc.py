"""ec_route_noalloc (routing with the library's static scratch array, for
callers that cannot allocate) against ec_route: the same scores, selection,
gates and slot map, bit for bit, on two calls in a row, the second with a
smaller problem and without a slot buffer (the slot map then also lives in the
scratch, which still holds the first call's transposed scores)."""
import numpy as np
import pytest
import torch

import paper_2604_01622_amd as ec
from paper_2604_01622_amd import synth

pytestmark = pytest.mark.gpu


def _dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(lens, d, E, seed, cf, dtype, with_slot):
    wl = synth.small(f"noalloc{seed}", lens, d, E, 64, dtype=dtype, seed=seed,
                     capacity_factor=cf)
    inp = synth.draw(wl)
    caps = ec.capacity(wl.group_lengths, E, c=cf)
    X, Wg = _dev(inp.X), _dev(inp.Wg)
    print(f"[case] noalloc lens={list(lens)[:3]}.. N={wl.n_tokens} d={d} E={E} {dtype} "
          f"slot={'given' if with_slot else 'scratch'}", flush=True)
    want = ec.route(X, Wg, wl.group_offsets, caps, 1.0, d_ff=64)
    got = ec.route_noalloc(X, Wg, wl.group_offsets, caps, 1.0, d_ff=64, with_slot=with_slot)
    torch.cuda.synchronize()
    for name, a, b in zip(("S", "sel_token", "sel_gate", "slot"), got, want):
        if a is None:
            continue
        assert torch.equal(a, b), name
    return got


def test_route_noalloc_matches_route_twice():
    # the benchmark's routing shape: 8 x 2048 tokens, 64 experts (4 MiB of scratch)
    _case([2048] * 8, 2048, 64, 60, 8.0, "bf16", True)
    # then a smaller ragged problem whose slot map also lives in the scratch
    _case([700, 333, 512], 256, 24, 61, 3.0, "bf16", False)


def test_route_noalloc_fp32_and_largest():
    # the largest problem the scratch holds without a slot buffer: E N 4 * 2 = 16 MiB
    _case([4096, 4096, 4096, 4096], 64, 128, 62, 8.0, "bf16", False)
    _case([300, 211], 128, 8, 63, 2.0, "f32", False)
