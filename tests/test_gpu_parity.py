"""Parity of the HIP path (through the C interface) with the CPU float64 oracle.

Tolerances (stated by the layer's specification, derived for fp32 storage):
  * scores S: max |S_gpu - S_ref| / S_ref <= 1e-5 (fp32 scores, fp32 accumulation);
  * selection: bit-exact against the oracle's selection run on the GPU's own S;
  * outputs and gradients: relative L2 <= 2e-2 for bf16 storage (fp32
    accumulation), <= 1e-4 for fp32 storage (fp32 sums of up to a few
    thousand terms, unit roundoff 6e-8).
"""
import os

import numpy as np
import pytest
import torch

from oracle import ec_ref as ref
import paper_2604_01622_amd as ec
from paper_2604_01622_amd import synth

pytestmark = pytest.mark.gpu

S_TOL = 1e-5
FP32_TINY = float(np.finfo(np.float32).tiny)


def out_tol(dtype):
    return 2e-2 if dtype == "bf16" else 1e-4


def dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def rel_l2(got, exp):
    got, exp = ref.widen(got), np.asarray(exp, dtype=np.float64)
    den = np.linalg.norm(exp)
    return float(np.linalg.norm(got - exp) / (den if den > 0 else 1.0))


def caps_for(wl, inp):
    """(library capacities, oracle capacities) for a workload; they must agree."""
    L = np.asarray(wl.group_lengths)
    if wl.time_dependent:
        k_lib = ec.capacity(L, wl.n_experts, t=inp.t, c_min=wl.c_min, c_max=wl.c_max)
        k_ref = ref.capacity_ref(L, wl.n_experts, t=inp.t, c_min=wl.c_min, c_max=wl.c_max)
    else:
        k_lib = ec.capacity(L, wl.n_experts, c=wl.capacity_factor)
        k_ref = ref.capacity_ref(L, wl.n_experts, c=wl.capacity_factor)
    assert np.array_equal(k_lib, k_ref)
    return k_lib


def check_route(inp, caps, inv_tau, S_rows=None):
    """Runs ec_route; checks S against the oracle (all rows or a sample) and the
    selection bit-exactly against the oracle run on the GPU's S."""
    wl = inp.wl
    off = wl.group_offsets
    X, Wg = dev(inp.X), dev(inp.Wg)
    S, sel, gate, slot = ec.route(X, Wg, off, caps, inv_tau, d_ff=wl.d_ff)
    torch.cuda.synchronize()
    S_h, sel_h, gate_h, slot_h = S.cpu().numpy(), sel.cpu().numpy(), gate.cpu().numpy(), slot.cpu().numpy()
    rows = np.arange(wl.n_tokens) if S_rows is None else S_rows
    S_ref = ref.router_ref(np.asarray(inp.X)[rows], inp.Wg, inv_tau)
    err = np.max(np.abs(S_h[rows].astype(np.float64) - S_ref) / S_ref) if len(rows) else 0.0
    assert err <= S_TOL, f"score error {err:.3g}"
    sel_ref = ref.select_ref(S_h.astype(np.float64), off, caps)
    assert sel_h.shape == sel_ref.shape
    assert np.array_equal(sel_h, sel_ref), "selection differs from the oracle on the GPU's scores"
    slot_exp = ref.slot_ref(sel_ref, wl.n_tokens).T
    assert np.array_equal(slot_h, slot_exp)
    if sel_h.size:
        assert np.array_equal(gate_h, np.take_along_axis(S_h.T, sel_h.astype(np.int64), 1))
    # token drop statistic from the slot map: exact counts
    cnt, dropped = ec.token_coverage(slot, off, caps)
    cnt_ref, dropped_ref = ref.coverage_ref(sel_ref, off)
    assert np.array_equal(cnt.cpu().numpy(), cnt_ref)
    assert np.array_equal(dropped.cpu().numpy(), dropped_ref)
    return S_h, sel_h


GRADS = ("dX", "dWg", "dW1", "dW3", "dW2")
SHARED_GRADS = ("dWs1", "dWs3", "dWs2")


def run_layer(inp, caps, inv_tau, backward=False):
    wl = inp.wl
    X, Wg, W1, W3, W2 = (dev(a) for a in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2))
    shared = None if inp.shared is None else tuple(dev(w) for w in inp.shared)
    Y, saved = ec.forward(X, Wg, W1, W3, W2, wl.group_offsets, caps, inv_tau, save=True,
                          shared=shared)
    out = {"Y": host(Y), "saved": saved}
    if backward:
        g = ec.backward(X, Wg, W1, W3, W2, dev(inp.dY), saved, wl.group_offsets, caps, inv_tau,
                        shared=shared)
        for n, t in zip(GRADS + (SHARED_GRADS if shared else ()), g):
            out[n] = host(t)
    torch.cuda.synchronize()
    P = ec.Problem.of(X, Wg, wl.d_ff, wl.group_offsets, caps, inv_tau, shared)
    out["views"] = {k: v for k, v in ec.saved_views(saved, P).items()}
    return out


def full_case(wl, inv_tau=None, backward=None, inp=None):
    inv_tau = wl.inv_temperatures[0] if inv_tau is None else inv_tau
    backward = wl.backward if backward is None else backward
    print(f"[case] {wl.name} inv_tau={inv_tau} backward={backward}", flush=True)
    inp = inp or synth.draw(wl, with_dy=backward)
    caps = caps_for(wl, inp)
    S_h, sel = check_route(inp, caps, inv_tau)
    out = run_layer(inp, caps, inv_tau, backward)
    # the forward's routing equals ec_route's (same kernels, deterministic)
    assert np.array_equal(out["views"]["sel_token"].cpu().numpy(), sel)
    assert np.array_equal(out["views"]["S"].cpu().numpy(), S_h)
    tol = out_tol(wl.dtype)
    args = (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2)
    sh = inp.shared
    if not backward:
        Y_ref = ref.forward_ref(*args, wl.group_offsets, caps, inv_tau, sel_token=sel,
                                shared=sh)["Y"]
        assert rel_l2(out["Y"], Y_ref) <= tol, rel_l2(out["Y"], Y_ref)
        return out
    g = ref.backward_ref(*args, inp.dY, wl.group_offsets, caps, inv_tau, sel_token=sel, shared=sh)
    Y_ref = ref.forward_ref(*args, wl.group_offsets, caps, inv_tau, sel_token=sel, shared=sh)["Y"]
    errs = {"Y": rel_l2(out["Y"], Y_ref)}
    for n in GRADS + (SHARED_GRADS if sh is not None else ()):
        errs[n] = rel_l2(out[n], g[n])
    print("[errs]", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(v <= tol for v in errs.values()), errs
    return out


# ------------------------------------------------------------------ small cases

def test_tiny_f32_forward_backward():
    wl = synth.TINY_F32
    full_case(wl, backward=True, inp=synth.draw(wl, with_dy=True))


RAGGED = dict(group_lengths=[700, 384, 530], d=256, E=16, h=320)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_multitile_forward_backward(dtype):
    wl = synth.small(f"ragged_{dtype}", RAGGED["group_lengths"], RAGGED["d"], RAGGED["E"],
                     RAGGED["h"], dtype=dtype, seed=11, c_min=4.0, c_max=12.0, backward=True)
    full_case(wl)


@pytest.mark.parametrize("inv_tau", [0.5, 2.0])
def test_temperature(inv_tau):
    wl = synth.small("temp", [512, 300], 128, 32, 128, seed=12, capacity_factor=3.0)
    full_case(wl, inv_tau=inv_tau)


@pytest.mark.parametrize("E", [1, 5, 17, 200, 256])
def test_expert_counts(E):
    wl = synth.small(f"E{E}", [256, 129], 128, E, 64, seed=13, capacity_factor=min(2.0, E))
    full_case(wl)


@pytest.mark.parametrize("dtype,d,h", [("bf16", 16384, 64), ("bf16", 64, 16384),
                                       ("f32", 16384, 64)])
def test_maximum_widths(dtype, d, h):
    # the widest model and hidden dimensions the interface accepts: 256 K-steps in
    # the products that contract over them, 2048 chunks per combine row
    wl = synth.small(f"wide_{dtype}_{d}_{h}", [130, 70], d, 3, h, dtype=dtype, seed=22,
                     capacity_factor=1.5, backward=True)
    full_case(wl)


@pytest.mark.parametrize("dtype,h", [("bf16", 512), ("bf16", 1024), ("bf16", 2048), ("f32", 256),
                                     ("f32", 1024), ("bf16", 768)])
def test_gate_gradient_partials(dtype, h):
    # the router backward sums each selected pair's gate-gradient partials (one per
    # 128 hidden units in bf16, 64 in fp32): 4, 8 and 16 per row read as vectors,
    # 6 through the general path
    wl = synth.small(f"dsp_{dtype}_{h}", [300, 157], 128, 16, h, dtype=dtype, seed=24,
                     capacity_factor=3.0, backward=True)
    full_case(wl)


@pytest.mark.parametrize("k", [100, 128, 257, 384, 385, 612])
def test_expert_buffer_row_counts(k):
    # expert buffers of k rows around the 256-row tile boundaries: one partial
    # block (100, 128), full blocks and a ragged last one (257, 384, 385, 612)
    wl = synth.small(f"rows{k}", [1024], 256, 4, 256, seed=25, capacity_factor=k / 256,
                     backward=True)
    inp = synth.draw(wl, with_dy=True)
    assert int(np.sum(caps_for(wl, inp))) == k
    full_case(wl, inp=inp)


def test_zero_capacity_everywhere():
    wl = synth.small("k0", [100, 50], 64, 8, 64, seed=14, capacity_factor=0.0, backward=True)
    out = full_case(wl)
    assert np.all(out["Y"] == 0) and np.all(out["dW1"] == 0) and np.all(out["dWg"] == 0)


def test_full_capacity_everywhere():
    # k = L: every expert takes every token of the group (dense soft mixture)
    wl = synth.small("kL", [96, 64], 128, 4, 128, seed=15, capacity_factor=4.0, backward=True)
    full_case(wl)


def test_empty_and_singleton_groups():
    wl = synth.small("empty", [0, 1, 300, 0, 77], 64, 8, 64, seed=16, capacity_factor=2.5,
                     backward=True)
    full_case(wl)


def test_many_groups():
    rng = np.random.default_rng(17)
    lens = rng.integers(5, 40, size=300)          # > one launch's group table
    wl = synth.small("many", lens, 64, 8, 64, seed=17, c_min=1.0, c_max=6.0)
    full_case(wl)


def test_many_tokens():
    # 64 sequences of 4096 tokens: 4096 router workgroups of 64 tokens, a top-k
    # grid of 16 x 64 columns, 32768 rows per expert buffer (128 row blocks)
    wl = synth.small("many_tokens", [4096] * 64, 128, 16, 128, seed=18, capacity_factor=2.0,
                     backward=True)
    full_case(wl)


def test_near_the_size_limit():
    # E K_tot 2 max(d, h) within 0.5% of the 2^31-element limit (the [E, K, 2h]
    # buffer of the backward: 4.3 GB; H1, H3 and A 2.1 GB each): sampled rows of
    # S, Y and dX, and sampled hidden units of every expert's weight gradients
    wl = synth.small("near_limit", [262112], 512, 2, 2048, seed=19, capacity_factor=1.99,
                     backward=True)
    print(f"[case] {wl.name}", flush=True)
    inp = synth.draw(wl, with_dy=True)
    caps = caps_for(wl, inp)
    K = int(np.sum(caps))
    assert 2 * K * 2 * 2048 < 2 ** 31 and 2 * K * 2 * 2048 > 0.99 * 2 ** 31
    rng = np.random.default_rng(19)
    rows = np.sort(rng.choice(wl.n_tokens, 48, replace=False))
    S_h, sel = check_route(inp, caps, 1.0, S_rows=rows)
    out = run_layer(inp, caps, 1.0, backward=True)
    assert np.array_equal(out["views"]["sel_token"].cpu().numpy(), sel)
    args = (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2)
    errs = {"Y": rel_l2(out["Y"][rows], ref.forward_rows_ref(*args, sel, rows, 1.0)),
            "dX": rel_l2(out["dX"][rows], ref.backward_rows_ref(*args, inp.dY, sel, rows, 1.0))}
    units = [0, 777, 2047]
    for j in range(2):
        g1, g3, g2 = ref.expert_grads_units_ref(*args, inp.dY, sel, j, units, 1.0)
        errs[f"dW1[{j}]"] = rel_l2(out["dW1"][j][units], g1)
        errs[f"dW3[{j}]"] = rel_l2(out["dW3"][j][units], g3)
        errs[f"dW2[{j}]"] = rel_l2(out["dW2"][j][:, units], g2)
    print("[errs]", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(v <= out_tol("bf16") for v in errs.values()), errs


def test_long_group_route_only():
    # a column longer than the LDS-cached top-k path
    wl = synth.small("long", [20000, 777], 64, 4, 64, seed=18, capacity_factor=1.5)
    inp = synth.draw(wl)
    caps = caps_for(wl, inp)
    check_route(inp, caps, 1.0)


@pytest.mark.parametrize("lens", [[500, 17], [2048, 1999, 64], [4096, 3000, 2049],
                                  [9000, 100], [13000, 5]])
@pytest.mark.parametrize("ties", [False, True])
def test_topk_every_path(lens, ties):
    """Every selection path: one wave per column with 8, 32 or 64 keys per lane
    (columns up to 512, 2048, 4096 tokens), then one workgroup per column with the
    keys cached in LDS (up to 12288) or re-read; normal scores and scores with
    whole runs of bitwise-equal values; capacities from 0 to the whole group."""
    wl = synth.small("paths", lens, 64, 8, 64, seed=23, capacity_factor=1.0)
    inp = synth.draw(wl)
    if ties:
        rng = np.random.default_rng(23)
        protos = rng.integers(-1, 2, size=(6, 64)).astype(np.float32)
        inp.X[:] = synth.f32_to_bf16_bits(protos[rng.integers(0, 6, size=wl.n_tokens)])
    rng = np.random.default_rng(24)
    caps = np.array([[0, 1, L // 3, L - 1, L][int(rng.integers(0, 5))] if L > 1 else L
                     for L in lens], dtype=np.int32)
    caps[0] = lens[0] // 8
    print(f"[case] top-k paths lens={lens} ties={ties} caps={caps.tolist()}", flush=True)
    check_route(inp, caps, 1.0)


def test_ties_zero_router():
    # Wg = 0: every score is exactly 1/E and each expert takes the first k tokens
    wl = synth.small("ties", [64, 40], 64, 8, 64, seed=19, capacity_factor=2.0)
    inp = synth.draw(wl)
    inp.Wg[:] = 0
    caps = caps_for(wl, inp)
    S_h, sel = check_route(inp, caps, 1.0)
    assert np.all(S_h == np.float32(1.0 / 8))
    exp = np.concatenate([np.arange(caps[0]), 64 + np.arange(caps[1])])
    assert np.array_equal(sel, np.tile(exp, (8, 1)))


def test_ties_repeated_tokens():
    # tokens drawn from 10 integer-valued prototypes: whole groups of tokens have
    # bitwise-equal scores, so every column's threshold falls inside a tie
    wl = synth.small("qties", [333, 200], 64, 8, 64, seed=20, capacity_factor=2.0)
    inp = synth.draw(wl)
    rng = np.random.default_rng(20)
    protos = rng.integers(-1, 2, size=(10, 64)).astype(np.float32)
    inp.X[:] = synth.f32_to_bf16_bits(protos[rng.integers(0, 10, size=wl.n_tokens)])
    inp.Wg[:] = synth.f32_to_bf16_bits(
        (rng.integers(-2, 3, size=inp.Wg.shape) / 8).astype(np.float32))
    caps = caps_for(wl, inp)
    S_h, sel = check_route(inp, caps, 1.0)
    assert len(np.unique(S_h[:, 0])) <= 10     # the ties are really there


def test_deterministic():
    wl = synth.small("det", [512, 512], 256, 16, 192, seed=21, capacity_factor=4.0, backward=True)
    inp = synth.draw(wl, with_dy=True)
    caps = caps_for(wl, inp)
    a = run_layer(inp, caps, 1.0, backward=True)
    b = run_layer(inp, caps, 1.0, backward=True)
    for n in ("Y", "dX", "dWg", "dW1", "dW3", "dW2"):
        assert np.array_equal(a[n], b[n]), n


def test_deterministic_full_training_step():
    """At the benchmark's size the training step gives bit-identical outputs on
    repeated runs (no atomics: every sum has a fixed order), and the inference
    forward agrees bit for bit with the training forward."""
    wl = synth.TRAIN_BF16
    print(f"[case] {wl.name} determinism", flush=True)
    inp = synth.draw(wl, with_dy=True)
    caps = caps_for(wl, inp)
    X, Wg, W1, W3, W2, dY = (dev(a) for a in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, inp.dY))
    layer = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, caps, wl.inv_temperatures[0],
                     training=True)
    runs = []
    for _ in range(2):
        y = layer.forward().clone()
        runs.append([y] + [t.clone() for t in layer.backward(dY)])
    torch.cuda.synchronize()
    for n, a, b in zip(("Y",) + GRADS, runs[0], runs[1]):
        assert torch.equal(a, b), n
    inf = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, caps, wl.inv_temperatures[0])
    assert torch.equal(inf.forward(), runs[0][0])


@pytest.mark.parametrize("dtype,shared", [("bf16", 0), ("bf16", 128), ("f32", 0)])
def test_graph_capture_replays(dtype, shared):
    """A training step captured in a HIP graph replays to the eager results bit
    for bit, replay after replay, with eager work between the replays (the
    library enqueues kernels only, no memory-set nodes)."""
    wl = synth.small("graph", [300, 212], 128, 8, 192, dtype=dtype, seed=44, capacity_factor=3.0,
                     backward=True, d_shared=shared)
    inp = synth.draw(wl, with_dy=True)
    caps = caps_for(wl, inp)
    X, Wg, W1, W3, W2, dY = (dev(a) for a in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, inp.dY))
    sh = None if inp.shared is None else tuple(dev(w) for w in inp.shared)
    layer = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, caps, 1.0, training=True, shared=sh)

    def step():
        y = layer.forward()
        return [y] + list(layer.backward(dY))

    eager = [t.clone() for t in step()]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = step()
    for r in range(3):
        for t in outs:
            t.zero_()   # eager work between replays; the replay must rewrite everything
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs, eager)):
            assert torch.equal(a, b), (r, i)


# ------------------------------------------------------------------ full-size workloads
# Same launch configuration as the benchmark; the oracle evaluates the whole
# layer: every row of S, every selected pair, every token's output, every
# gradient element, and each expert's outputs and weight gradients separately
# (the worst expert is printed and must meet the bound too).

def _per_expert(name, got, errs, worst):
    """Returns a callback for the oracle's per-expert outputs that records the
    relative L2 error of expert j's rows of `got` [E, K, d]."""
    def cb(j, o):
        e = rel_l2(got[j], o)
        if e > worst.get(name, (-1.0, -1))[0]:
            worst[name] = (e, j)
    return cb


def _report(errs, worst, tol=2e-2):
    print("[errs]", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    print("[worst expert]", {k: f"{v[0]:.2e} (expert {v[1]})" for k, v in worst.items()},
          flush=True)
    assert all(v <= tol for v in errs.values()), errs
    assert all(v[0] <= tol for v in worst.values()), worst


def _full_forward(wl, inv_tau):
    print(f"[case] {wl.name} inv_tau={inv_tau}", flush=True)
    inp = synth.draw(wl)
    caps = caps_for(wl, inp)
    print(f"[caps] {[int(k) for k in caps]}", flush=True)
    S_h, sel = check_route(inp, caps, inv_tau)            # every row of S
    out = run_layer(inp, caps, inv_tau)                   # training forward (saves O)
    assert np.array_equal(out["views"]["sel_token"].cpu().numpy(), sel)
    # the inference forward (the benchmark's launch) equals the training forward
    X, Wg, W1, W3, W2 = (dev(a) for a in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2))
    Y_inf = host(ec.forward(X, Wg, W1, W3, W2, wl.group_offsets, caps, inv_tau))
    assert np.array_equal(Y_inf, out["Y"])
    O = host(out["views"]["O"])
    errs, worst = {}, {}
    Y_ref = ref.forward_ref(inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, wl.group_offsets, caps,
                            inv_tau, sel_token=sel,
                            on_expert=_per_expert("O", O, errs, worst))["Y"]
    errs["Y"] = rel_l2(out["Y"], Y_ref)
    unsel = np.setdiff1d(np.arange(wl.n_tokens), np.unique(sel))
    assert np.all(out["Y"][unsel] == 0)
    _report(errs, worst)


def test_full_static_bf16():
    _full_forward(synth.STATIC_BF16, 1.0)


def test_full_timestep_bf16():
    _full_forward(synth.TIMESTEP_BF16, 1.0)


@pytest.mark.parametrize("inv_tau", synth.FINE_BF16.inv_temperatures)
def test_full_fine_bf16(inv_tau):
    _full_forward(synth.FINE_BF16, inv_tau)


def test_full_decode_bf16():
    # single-sample decoding: one routing group, every expert picks from its 2048 tokens
    _full_forward(synth.DECODE_BF16, 1.0)


def _full_train(wl):
    print(f"[case] {wl.name} backward", flush=True)
    inp = synth.draw(wl, with_dy=True)
    caps = caps_for(wl, inp)
    S_h, sel = check_route(inp, caps, 1.0)
    out = run_layer(inp, caps, 1.0, backward=True)
    O = host(out["views"]["O"])
    errs, worst = {}, {}
    g = ref.backward_ref(inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, inp.dY, wl.group_offsets, caps,
                         1.0, sel_token=sel, shared=inp.shared,
                         on_expert=_per_expert("O", O, errs, worst))
    names = GRADS + (SHARED_GRADS if inp.shared is not None else ())
    errs["Y"] = rel_l2(out["Y"], g["Y"])
    for n in names:
        errs[n] = rel_l2(out[n], g[n])
    for n in ("dW1", "dW3", "dW2"):
        for j in range(wl.n_experts):
            e = rel_l2(out[n][j], g[n][j])
            if e > worst.get(n, (-1.0, -1))[0]:
                worst[n] = (e, j)
    _report(errs, worst)


def test_full_train_bf16():
    _full_train(synth.TRAIN_BF16)


# ------------------------------------------------------------------ saved activations

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_saved_activations_carry_the_gate(dtype):
    """The saved buffer holds what the header documents: sel_gate is S at the
    selection (an exact copy), A = gate * SiLU(H1) * H3 and O = A W2^T, checked
    against the saved H1, H3 and A themselves (so only the epilogue's arithmetic
    and the product are under test)."""
    wl = synth.small(f"gate_{dtype}", [300, 200], 128, 8, 192, dtype=dtype, seed=5,
                     capacity_factor=3.0)
    print(f"[case] saved activations {dtype}", flush=True)
    inp = synth.draw(wl)
    caps = caps_for(wl, inp)
    v = run_layer(inp, caps, wl.inv_temperatures[0])["views"]
    S, sel = v["S"].cpu().numpy(), v["sel_token"].cpu().numpy()
    g = v["sel_gate"].cpu().numpy()
    assert np.array_equal(g, S[sel, np.arange(wl.n_experts)[:, None]])
    H1, H3, A = (ref.widen(host(v[n])) for n in ("H1", "H3", "A"))
    A_exp = g[..., None].astype(np.float64) * (H1 / (1.0 + np.exp(-H1))) * H3
    tol = out_tol(wl.dtype)
    assert rel_l2(A, A_exp) <= tol, rel_l2(A, A_exp)
    O_exp = np.matmul(A, np.swapaxes(ref.widen(inp.W2), 1, 2))
    assert rel_l2(host(v["O"]), O_exp) <= tol, rel_l2(host(v["O"]), O_exp)


# ------------------------------------------------------------------ K-major operands

@pytest.mark.parametrize("groups,d,h,cf", [
    ([300], 192, 320, 4.0),        # ragged column blocks; the W1 | W3 split inside a tile
    ([900, 650], 64, 192, 8.0),    # more row blocks than k-steps
    ([2048], 256, 128, 12.0),      # twelve row blocks share four k-steps
])
def test_kmajor_weights_and_gathered_rows(groups, d, h, cf):
    """The backward reads the expert weights K-major (dA: W2, dX: W1 then W3
    along one contraction) and its weight-gradient products gather the rows of
    X and dY per k row; the training forward saves no gathered or transposed
    copies (bf16)."""
    wl = synth.small("km", groups, d, 8, h, seed=43, capacity_factor=cf, d_shared=128,
                     backward=True)
    print(f"[case] K-major groups={groups} d={d} h={h} cf={cf}", flush=True)
    out = full_case(wl)
    assert "Xe" not in out["views"]


# ------------------------------------------------------------------ shared experts

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_shared_experts_forward_backward(dtype):
    # 777 tokens: the shared weight gradients' split over the tokens ends in a short split
    wl = synth.small("shared", [500, 277], 128, 8, 192, dtype=dtype, seed=40, c_min=1.0,
                     c_max=3.0, backward=True, d_shared=256)
    full_case(wl)


def test_shared_experts_without_routed_capacity():
    # no routed expert takes any token: the layer is the shared SwiGLU alone
    wl = synth.small("shared0", [200, 56], 64, 4, 64, seed=41, capacity_factor=0.0,
                     backward=True, d_shared=128)
    out = full_case(wl)
    assert np.all(out["dW1"] == 0) and np.all(out["dW2"] == 0)


def test_full_train_shared_bf16():
    _full_train(synth.TRAIN_SHARED_BF16)


# ------------------------------------------------------------------ token choice (comparison policy)

def check_tc(inp, caps, top_k, inv_tau=1.0, y_rows=None, S_rows=None):
    """Token-choice routing and forward through the C interface: scores, the kept
    pairs (bit-exact against the oracle's selection on the GPU's scores), the
    packed layout, the gates, and the layer output."""
    wl = inp.wl
    off = wl.group_offsets
    X, Wg, W1, W3, W2 = (dev(a) for a in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2))
    S, G, slot, rows, sel = ec.tc_route(X, Wg, off, caps, top_k, inv_tau, d_ff=wl.d_ff)
    Y, rows2 = ec.tc_forward(X, Wg, W1, W3, W2, off, caps, top_k, inv_tau)
    torch.cuda.synchronize()
    S_h, G_h, slot_h = S.cpu().numpy(), G.cpu().numpy(), slot.cpu().numpy()
    rows_h, sel_h = rows.cpu().numpy(), sel.cpu().numpy()
    assert np.array_equal(rows_h, rows2.cpu().numpy())
    srows = np.arange(wl.n_tokens) if S_rows is None else S_rows
    S_ref = ref.router_ref(np.asarray(inp.X)[srows], inp.Wg, inv_tau)
    # relative error, with an absolute floor at fp32's smallest normal number
    # (scores below it cannot carry a relative precision in fp32)
    dS = np.abs(S_h[srows].astype(np.float64) - S_ref)
    assert np.all(dS <= S_TOL * S_ref + FP32_TINY)
    choice, gate, kept, trows = ref.tc_select_ref(S_h.astype(np.float64), off, top_k, caps)
    # packed layout: expert j's kept tokens, ascending, at rows [rows[j], rows[j+1])
    want_rows = np.concatenate([[0], np.cumsum([len(r) for r in trows])])
    assert np.array_equal(rows_h, want_rows)
    for j in range(wl.n_experts):
        seg = np.arange(want_rows[j], want_rows[j + 1])
        assert np.array_equal(sel_h[seg], trows[j])
        exp_slot = np.full(wl.n_tokens, -1)
        exp_slot[trows[j]] = seg
        assert np.array_equal(slot_h[j], exp_slot)
    # gates of the kept pairs; zero elsewhere
    Gw = np.zeros_like(G_h, dtype=np.float64)
    for r in range(top_k):
        Gw[np.arange(wl.n_tokens), choice[:, r]] += np.where(kept[:, r], gate[:, r], 0.0)
    assert np.array_equal(G_h != 0, Gw != 0)
    nz = Gw != 0
    assert np.max(np.abs(G_h[nz] - Gw[nz]) / Gw[nz]) <= 1e-6
    Yh = host(Y)
    if y_rows is None:
        Y_ref = ref.tc_forward_ref(inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, off, top_k, caps,
                                   inv_tau, selection=(choice, kept))["Y"]
        err = rel_l2(Yh, Y_ref)
    else:
        Y_ref = ref.tc_forward_rows_ref(inp.X, inp.Wg, inp.W1, inp.W3, inp.W2, choice, kept,
                                        y_rows, inv_tau)
        err = rel_l2(Yh[y_rows], Y_ref)
    print(f"[errs] tc Y {err:.2e}; kept {kept.sum()} of {kept.size} pairs; "
          f"loads max/mean {np.diff(rows_h).max() / max(np.diff(rows_h).mean(), 1e-9):.2f}",
          flush=True)
    assert err <= out_tol(wl.dtype), err
    return rows_h, kept


@pytest.mark.parametrize("top_k,cf", [(2, 1.0), (2, 0.0), (8, 0.0)])
def test_tc_ragged_bf16(top_k, cf):
    wl = synth.small("tc", [300, 212], 128, 8, 192, seed=50, capacity_factor=1.0)
    inp = synth.draw(wl)
    caps = ec.tc_capacity(wl.group_lengths, 8, top_k, cf)
    assert np.array_equal(caps, ref.tc_capacity_ref(wl.group_lengths, 8, top_k, cf))
    rows, kept = check_tc(inp, caps, top_k)
    if cf > 0:
        assert not kept.all()            # the cap drops pairs in this case


def test_tc_top1_odd_experts():
    wl = synth.small("tc1", [257, 100], 64, 17, 64, seed=51, capacity_factor=1.0)
    inp = synth.draw(wl)
    check_tc(inp, ec.tc_capacity(wl.group_lengths, 17, 1, 1.25), 1)


def test_tc_f32():
    wl = synth.small("tcf", [128, 70], 64, 8, 128, dtype="f32", seed=52, capacity_factor=1.0)
    inp = synth.draw(wl)
    check_tc(inp, ec.tc_capacity(wl.group_lengths, 8, 2, 1.0), 2)


def test_tc_skewed_router_with_empty_experts():
    # router rows of very different norms: a few experts take most tokens and
    # some none at all (zero-row experts in the grouped GEMM)
    wl = synth.small("tcskew", [400, 300], 128, 16, 128, seed=53, capacity_factor=1.0)
    inp = synth.draw(wl)
    rng = np.random.default_rng(53)
    scale = np.exp(rng.normal(0.0, 1.0, size=(16, 1)))
    scale[[3, 9]] = 1e-3
    inp.Wg[:] = synth.f32_to_bf16_bits((ref.widen(inp.Wg) * scale * 3).astype(np.float32))
    for cf in (0.0, 1.0):
        rows, kept = check_tc(inp, ec.tc_capacity(wl.group_lengths, 16, 2, cf), 2)
        if cf == 0:
            assert np.any(np.diff(rows) == 0)


@pytest.mark.parametrize("E,top_k,zero_router", [(65, 3, False), (200, 7, False), (256, 256, False),
                                                 (64, 8, True), (130, 5, True)])
def test_tc_expert_counts_and_ties(E, top_k, zero_router):
    # the row top-k keeps a token's scores in 16 lanes (4 or 16 experts a lane);
    # a zero router makes every score equal, so each token takes the lowest
    # expert indices
    wl = synth.small(f"tcE{E}", [200, 77], 64, E, 64, seed=54, capacity_factor=1.0)
    inp = synth.draw(wl)
    if zero_router:
        inp.Wg[:] = 0
    rows, kept = check_tc(inp, ec.tc_capacity(wl.group_lengths, E, top_k, 1.0), top_k)
    if zero_router:
        assert np.all(np.diff(rows)[top_k:] == 0)


def test_full_tc_timestep_bf16():
    wl = synth.TIMESTEP_BF16
    print(f"[case] token choice on {wl.name}", flush=True)
    inp = synth.draw(wl)
    for cf in (1.0, 0.0):
        caps = ec.tc_capacity(wl.group_lengths, wl.n_experts, 8, cf)
        check_tc(inp, caps, 8)


# ------------------------------------------------------------------ randomised shapes

# EC_RANDOM_CASES / EC_RANDOM_TC_CASES widen the sweeps (defaults 8 and 4)
@pytest.mark.parametrize("seed", range(int(os.environ.get("EC_RANDOM_CASES", "8"))))
def test_random_problems(seed):
    rng = np.random.default_rng(1000 + seed)
    G = int(rng.integers(1, 5))
    lens = [int(x) for x in rng.integers(0, 500, size=G)]
    if sum(lens) == 0:
        lens[0] = 7
    d = 64 * int(rng.integers(1, 7))
    E = int(rng.integers(1, 41))
    h = 64 * int(rng.integers(1, 7))
    dtype = "f32" if seed % 4 == 3 else "bf16"
    d_shared = 64 * int(rng.integers(0, 4))
    if rng.random() < 0.5:
        kw = dict(capacity_factor=float(rng.uniform(0.5, 4.0)))
    else:
        kw = dict(c_min=float(rng.uniform(0.5, 2.0)), c_max=float(rng.uniform(2.0, 6.0)))
    wl = synth.small(f"rnd{seed}", lens, d, E, h, dtype=dtype, seed=2000 + seed, backward=True,
                     inv_temperature=float(rng.choice([0.5, 1.0, 2.0])), d_shared=d_shared, **kw)
    print(f"[case] lens={lens} d={d} E={E} h={h} {dtype} shared={d_shared} {kw}", flush=True)
    full_case(wl)


# larger shapes: several row blocks per expert buffer, the 192-row tiles, every
# column top-k variant, up to 256 experts (EC_RANDOM_LARGE_CASES widens it)
@pytest.mark.parametrize("seed", range(int(os.environ.get("EC_RANDOM_LARGE_CASES", "2"))))
def test_random_large_problems(seed):
    rng = np.random.default_rng(5000 + seed)
    G = int(rng.integers(1, 4))
    lens = [int(x) for x in rng.integers(1, 4500, size=G)]
    E = int(rng.choice([8, 33, 64, 128, 256]))
    d = 64 * int(rng.integers(4, 17))
    h = 64 * int(rng.integers(2, 13))
    backward = bool(rng.random() < 0.5)
    kw = dict(c_min=float(rng.uniform(0.5, 2.0)), c_max=float(rng.uniform(2.0, 8.0)))
    wl = synth.small(f"rndL{seed}", lens, d, E, h, seed=6000 + seed, backward=backward,
                     inv_temperature=float(rng.choice([0.5, 1.0, 2.0])), **kw)
    print(f"[case] lens={lens} d={d} E={E} h={h} backward={backward} {kw}", flush=True)
    full_case(wl)


@pytest.mark.parametrize("seed", range(int(os.environ.get("EC_RANDOM_TC_CASES", "4"))))
def test_random_token_choice(seed):
    rng = np.random.default_rng(3000 + seed)
    lens = [int(x) for x in rng.integers(1, 400, size=int(rng.integers(1, 4)))]
    d, h = 64 * int(rng.integers(1, 5)), 64 * int(rng.integers(1, 5))
    E = int(rng.integers(2, 33))
    k = int(rng.integers(1, min(E, 8) + 1))
    cf = float(rng.choice([0.0, 1.0, 1.5]))
    wl = synth.small(f"tcrnd{seed}", lens, d, E, h, seed=4000 + seed, capacity_factor=1.0)
    print(f"[case] tc lens={lens} d={d} E={E} h={h} k={k} cf={cf}", flush=True)
    check_tc(synth.draw(wl), ec.tc_capacity(lens, E, k, cf), k)
