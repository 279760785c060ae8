"""Host-side checks of the C interface (no GPU needed): the library loads and
exports every function the header declares, argument validation rejects bad
calls before anything is enqueued, and the host capacity rule agrees with the
oracle's."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

from oracle import ec_ref as ref
import paper_2604_01622_amd as ec
from paper_2604_01622_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ec_moe.h")

EC_OK, EC_ERR_ARG, EC_ERR_SHAPE, EC_ERR_CAPACITY, EC_ERR_DTYPE, EC_ERR_ALIGN, EC_ERR_WORKSPACE = range(7)


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ec_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    L = ec.lib()
    names = header_functions()
    assert set(names) == set(binding.EXPORTS), names
    for n in names:
        assert hasattr(L, n), n
    assert L.ec_status_string(EC_ERR_CAPACITY).decode().startswith("EC_ERR_CAPACITY")


def _problem(**kw):
    args = dict(n_tokens=256, d_model=128, n_experts=8, d_ff=64, group_offsets=[0, 100, 256],
                capacity=[10, 20], inv_temperature=1.0, dtype=torch.bfloat16)
    args.update(kw)
    return binding.Problem(**args)


FAKE = ctypes.c_void_p(1 << 20)       # aligned, never dereferenced: validation fails first
MISALIGNED = ctypes.c_void_p((1 << 20) + 8)


def _route(P, X=FAKE, ws_bytes=1 << 30):
    L = ec.lib()
    return L.ec_route(P.ref, X, FAKE, FAKE, FAKE, None, None, FAKE, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(capacity=[101, 20]), EC_ERR_CAPACITY),
    (dict(capacity=[-1, 20]), EC_ERR_CAPACITY),
    (dict(n_tokens=255), EC_ERR_SHAPE),                       # N != off[G]
    (dict(group_offsets=[0, 300, 256]), EC_ERR_SHAPE),        # decreasing offsets
    (dict(group_offsets=[1, 100, 256]), EC_ERR_SHAPE),
    (dict(d_model=100), EC_ERR_SHAPE),
    (dict(d_ff=32), EC_ERR_SHAPE),
    (dict(n_experts=0), EC_ERR_SHAPE),
    (dict(n_experts=257), EC_ERR_SHAPE),
    (dict(inv_temperature=0.0), EC_ERR_ARG),
    (dict(d_shared=32), EC_ERR_SHAPE),
    (dict(d_shared=96), EC_ERR_SHAPE),
    (dict(d_shared=-64), EC_ERR_SHAPE),
    (dict(inv_temperature=float("nan")), EC_ERR_ARG),
])
def test_invalid_problems_rejected(kw, status):
    P = _problem(**kw)
    assert _route(P) == status
    assert ec.lib().ec_last_error().decode() != ""
    assert ec.lib().ec_workspace_size(P.ref, 1) == 0
    assert ec.lib().ec_total_capacity(P.ref) == -1


def test_bad_dtype_and_pointers():
    P = _problem()
    P.c.dtype = 7
    assert _route(P) == EC_ERR_DTYPE
    P = _problem()
    assert _route(P, X=None) == EC_ERR_ARG
    assert _route(P, X=MISALIGNED) == EC_ERR_ALIGN
    assert _route(P, ws_bytes=16) == EC_ERR_WORKSPACE
    L = ec.lib()
    # forward: saved buffer too small, workspace too small
    NS = (None, None, None)          # no shared experts
    st = L.ec_moe_forward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, FAKE, 64, FAKE, 1 << 40,
                          None)
    assert st == EC_ERR_WORKSPACE
    st = L.ec_moe_forward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, None, 0, FAKE, 64, None)
    assert st == EC_ERR_WORKSPACE
    # shared experts declared but their weights missing
    Ps = _problem(d_shared=128)
    st = L.ec_moe_forward(Ps.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, None, 0, FAKE, 1 << 40,
                          None)
    assert st == EC_ERR_ARG
    # backward needs the saved buffer
    st = L.ec_moe_backward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, None, 0, FAKE, FAKE,
                           FAKE, FAKE, FAKE, *NS, FAKE, 1 << 40, None)
    assert st == EC_ERR_ARG
    assert L.ec_workspace_size(P.ref, 9) == 0


def test_token_coverage_validation():
    L = ec.lib()
    P = _problem()
    assert L.ec_token_coverage(P.ref, FAKE, FAKE, None, None) == EC_ERR_ARG        # dropped
    assert L.ec_token_coverage(P.ref, None, FAKE, FAKE, None) == EC_ERR_ARG        # slot, N > 0
    assert L.ec_token_coverage(P.ref, FAKE, MISALIGNED, FAKE, None) == EC_ERR_ALIGN
    assert L.ec_token_coverage(_problem(capacity=[101, 20]).ref, FAKE, FAKE, FAKE,
                               None) == EC_ERR_CAPACITY


def test_workspace_and_saved_layout():
    P = _problem()
    assert P.K == 30
    lay = P.saved_layout()
    order = ["S", "sel_token", "sel_gate", "slot", "H1", "H3", "A", "O", "total"]
    offs = [lay[k] for k in order]
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
    N, E, K, d, h = 256, 8, 30, 128, 64
    assert lay["sel_token"] - lay["S"] >= N * E * 4
    assert lay["sel_gate"] - lay["sel_token"] >= E * K * 4 and lay["slot"] - lay["sel_gate"] >= E * K * 4
    assert lay["H1"] - lay["slot"] >= E * N * 4
    assert lay["Xe"] == lay["total"]     # bf16 gathers the selected rows inside the products
    assert lay["total"] - lay["O"] >= E * K * d * 2
    for mode in (0, 1, 2, 3):
        assert P.workspace_size(mode) > 0
    assert P.saved_size() == lay["total"]
    assert lay["Hs1"] == lay["Hs3"] == lay["As"] == lay["total"]    # no shared experts
    Ps = _problem(d_shared=192)
    ls = Ps.saved_layout()
    assert [ls[k] for k in order[:8]] == offs[:8]
    assert ls["Hs3"] - ls["Hs1"] >= N * 192 * 2 and ls["As"] - ls["Hs3"] >= N * 192 * 2
    assert ls["total"] - ls["As"] >= N * 192 * 2
    assert Ps.workspace_size(1) > P.workspace_size(1) and Ps.workspace_size(2) > P.workspace_size(2)
    lf = _problem(dtype=torch.float32).saved_layout()
    assert lf["H1"] - lf["Xe"] >= E * K * d * 4 and lf["Xe"] - lf["slot"] >= E * N * 4


@pytest.mark.parametrize("sched", list(binding.SCHEDULERS))
def test_capacity_rule_matches_oracle(sched):
    rng = np.random.default_rng(3)
    lens = rng.integers(0, 5000, size=64)
    t = rng.uniform(0, 1, size=64)
    t[:4] = [0.0, 1.0, 0.5, 0.25]
    got = ec.capacity(lens, 64, t=t, c_min=4.0, c_max=12.0, scheduler=sched)
    exp = ref.capacity_ref(lens, 64, t=t, c_min=4.0, c_max=12.0, sched=sched)
    assert np.array_equal(got, exp)
    got = ec.capacity(lens, 64, c=8.0)
    assert np.array_equal(got, ref.capacity_ref(lens, 64, c=8.0))
    # half-to-even on exact ties: L c / E = 2.5 -> 2 and 3.5 -> 4
    assert list(ec.capacity([5, 7], 2, c=1.0)) == [2, 4]


@pytest.mark.parametrize("k,cf", [(8, 1.0), (8, 1.25), (2, 0.0), (1, 1.5), (4, 3.0)])
def test_tc_capacity_matches_oracle(k, cf):
    L = [2048, 100, 7, 0, 513]
    assert np.array_equal(ec.tc_capacity(L, 64 if k == 8 else 8, k, cf),
                          ref.tc_capacity_ref(L, 64 if k == 8 else 8, k, cf))


def test_tc_validation():
    L = ec.lib()
    P = _problem()
    ws = 1 << 30
    assert L.ec_tc_route(P.ref, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, None) == EC_ERR_ARG
    assert L.ec_tc_route(P.ref, 9, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, None) == EC_ERR_ARG
    assert L.ec_tc_route(P.ref, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, ws, None) == EC_ERR_ARG
    assert L.ec_tc_route(P.ref, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, None) == EC_ERR_WORKSPACE
    assert L.ec_tc_workspace_size(P.ref, 2, 0) > 0
    assert L.ec_tc_workspace_size(P.ref, 2, 1) > L.ec_tc_workspace_size(P.ref, 2, 0)
    assert L.ec_tc_workspace_size(P.ref, 0, 1) == 0
    st = L.ec_tc_forward(P.ref, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, FAKE, None,
                         FAKE, 64, None)
    assert st == EC_ERR_WORKSPACE


def test_forward_workspace_with_saved_buffer():
    """With a saved buffer the forward's activations live there, so its workspace
    (mode 3) holds only the transposed scores; without one (mode 1) the
    workspace also carries S, the selection, the slot map, A and O."""
    L = ec.lib()
    N, E, K, d, h = 256, 8, 30, 128, 64
    P = _problem()
    w1, w3 = P.workspace_size(1), P.workspace_size(3)
    assert w3 == -(-E * N * 4 // 256) * 256                # ST only
    assert w1 - w3 >= N * E * 4 + 2 * E * K * 4 + E * N * 4 + E * K * (h + d) * 2
    # the benchmark's training shapes: about 0.88 GB smaller
    big = binding.Problem(16384, 2048, 64, 1024, [0] + [2048 * (g + 1) for g in range(8)],
                          [278, 182, 362, 269, 350, 139, 338, 289], 1.0, torch.bfloat16)
    assert big.workspace_size(1) - big.workspace_size(3) > 0.85e9
    NS = (None, None, None)
    sv = P.saved_size()
    # with a saved buffer, a mode-3 workspace is enough; one byte less is rejected
    st = L.ec_moe_forward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, FAKE, sv, FAKE, w3 - 1,
                          None)
    assert st == EC_ERR_WORKSPACE
    # without a saved buffer, the mode-3 size is too small
    st = L.ec_moe_forward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, None, 0, FAKE, w3, None)
    assert st == EC_ERR_WORKSPACE
    assert "workspace" in L.ec_last_error().decode()
    # a saved buffer one byte short is rejected before the workspace is looked at
    st = L.ec_moe_forward(P.ref, FAKE, FAKE, FAKE, FAKE, FAKE, *NS, FAKE, FAKE, sv - 1, FAKE, w1,
                          None)
    assert st == EC_ERR_WORKSPACE and "saved" in L.ec_last_error().decode()
    assert L.ec_saved_size(_problem(capacity=[101, 20]).ref) == 0


def test_route_noalloc_rejects_problems_beyond_its_scratch():
    """Validation happens on the host before any HIP call: a problem whose
    transposed scores (E N 4 bytes, twice that without a slot buffer) exceed the
    static scratch is refused with EC_ERR_WORKSPACE."""
    L = ec.lib()
    limit = 16 << 20
    # E N 4 = 16 MiB: fits with a slot buffer, not without one
    P = binding.Problem(32768, 64, 128, 64, [0, 32768], [256], 1.0, torch.bfloat16)
    st = L.ec_route_noalloc(P.ref, FAKE, FAKE, FAKE, FAKE, None, None, None)
    assert st == EC_ERR_WORKSPACE and str(limit) in L.ec_last_error().decode()
    P2 = binding.Problem(32769, 64, 128, 64, [0, 32769], [256], 1.0, torch.bfloat16)
    st = L.ec_route_noalloc(P2.ref, FAKE, FAKE, FAKE, FAKE, None, FAKE, None)
    assert st == EC_ERR_WORKSPACE
    # the usual argument checks come first
    assert L.ec_route_noalloc(_problem(capacity=[101, 20]).ref, FAKE, FAKE, FAKE, FAKE, None,
                              None, None) == EC_ERR_CAPACITY
    assert L.ec_route_noalloc(_problem().ref, MISALIGNED, FAKE, FAKE, FAKE, None, None,
                              None) == EC_ERR_ALIGN


def test_product_path_fails_loudly_without_the_library(monkeypatch, tmp_path):
    # no CPU fallback: every entry point needs the built HIP library
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "libecmoe.so"))
    with pytest.raises(RuntimeError, match="missing"):
        binding.capacity([2048], 64, c=8.0)
    X = torch.zeros((16, 64), dtype=torch.bfloat16)
    Wg = torch.zeros((4, 64), dtype=torch.bfloat16)
    with pytest.raises(RuntimeError, match="missing"):
        binding.route(X, Wg, [0, 16], [4], 1.0)
