"""CPU float64 oracle of the expert-choice (EC) MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, links or calls
this module: only the tests, the smoke check and the CPU-baseline leg of the
benchmark do.  It shares no code with the HIP library.

Every function evaluates the plain definition in float64 on the exact stored
input values (bf16 bit patterns or fp32 values widened to float64).  Matrix
products use numpy's matmul as a library primitive; there is no blocking or
fusion beyond the definitions below.

Notation (the letters of the layer's interface; the paper swaps c and k between
its Section 2.2 and its Section 4):
  N tokens, d model width, E experts, h expert hidden width,
  G routing groups (sequences), group g = tokens [off[g], off[g+1]),
  k_g tokens selected by each expert in group g,
  c capacity factor (average experts per token, c = k*E/L),
  t mask ratio of a sequence.

Pins (tests/test_oracle.py): brute-force selection on tiny inputs, exactly k_g
tokens per (group, expert), softmax closed forms, the dense soft mixture when
every token is selected, the textbook SwiGLU FFN when E = 1, central finite
differences and torch autograd of the backward, Table 5 of the paper for the
capacity schedulers and Figure 2's per-expert loads, the drop statistic's
closed cases (every token kept when k_g = L_g, every token dropped when
k_g = 0, L_g - k_g dropped when E = 1), and for token choice the rank
definition of the row top-k with ties, first-come capacity, the arg-max expert
at top-1, the expert-choice mixture at top-E without a cap, and the
dropped-pair gate rule against a construction from torch's stable sort.
Mutation tests plant plausible mistakes (tie direction, temperature, the
activation, W1 and W3 swapped, a dropped softmax-Jacobian term) and check that
a pin fails.
"""
from __future__ import annotations

import itertools
import math

import numpy as np


# ---------------------------------------------------------------------------
# Storage formats
# ---------------------------------------------------------------------------

def widen(a: np.ndarray) -> np.ndarray:
    """Exact float64 value of stored data: uint16 arrays are bf16 bit patterns."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ---------------------------------------------------------------------------
# Capacity (Section 4.2 capacity function, Table 1 schedulers, Appendix H)
# ---------------------------------------------------------------------------

GAUSS_SIGMA = 0.22  # Appendix H


def gaussian_g(r, sigma: float = GAUSS_SIGMA):
    """Unnormalised bump exp(-(r - 1/2)^2 / (2 sigma^2)) of the Gaussian scheduler (Appendix H)."""
    r = np.asarray(r, dtype=np.float64)
    return np.exp(-((r - 0.5) ** 2) / (2.0 * sigma * sigma))


def gaussian_g_tilde(r, sigma: float = GAUSS_SIGMA):
    """Gaussian rescaled so that it is 0 at r = 0 and r = 1 and 1 at r = 1/2 (Appendix H)."""
    g0 = math.exp(-1.0 / (8.0 * sigma * sigma))
    return (gaussian_g(r, sigma) - g0) / (1.0 - g0)


def scheduler(name: str, r):
    """Scheduler s(r) in [0, 1] of Table 1 as a function of the mask ratio r."""
    r = np.asarray(r, dtype=np.float64)
    if name == "linear":
        return r.copy()
    if name == "linear_rev":
        return 1.0 - r
    if name == "cosine":
        return 0.5 * (1.0 - np.cos(np.pi * r))
    if name == "cosine_rev":
        return 0.5 * (1.0 + np.cos(np.pi * r))
    if name == "gaussian":
        return gaussian_g_tilde(r)
    if name == "gaussian_rev":
        return 1.0 - gaussian_g_tilde(r)
    raise ValueError(f"unknown scheduler {name!r}")


def capacity_factor_ref(t, c_min: float, c_max: float, sched: str = "linear_rev"):
    """c(t) = clamp(c_min + (c_max - c_min) s(t), c_min, c_max)  (Section 4.2)."""
    c = c_min + (c_max - c_min) * scheduler(sched, t)
    return np.clip(c, c_min, c_max)


def capacity_ref(group_lengths, n_experts: int, c=None, t=None, c_min=None, c_max=None,
                 sched: str = "linear_rev") -> np.ndarray:
    """Tokens per expert in each group.

    Section 2.2 equates expert-choice capacity with a token-choice top-c budget:
    E experts taking k tokens each out of L give E*k = c*L pairs, so k = L*c/E.  With a time-dependent capacity,
    c = c(t_g) per group (Section 4.2).  k is rounded half-to-even and clamped to
    [0, L_g].
    """
    L = np.asarray(group_lengths, dtype=np.float64)
    if c is not None:
        cg = np.full(L.shape, float(c))
    else:
        cg = capacity_factor_ref(np.asarray(t, dtype=np.float64), c_min, c_max, sched)
    k = np.rint(L * cg / float(n_experts))
    return np.clip(k, 0, L).astype(np.int64)


# ---------------------------------------------------------------------------
# Router (Section 2.2: score matrix S in R^{N x E}; softmax over the experts)
# ---------------------------------------------------------------------------

def softmax_ref(Z: np.ndarray, inv_tau: float = 1.0) -> np.ndarray:
    """Row softmax of Z / tau, shifted by the row maximum for stability."""
    Z = np.asarray(Z, dtype=np.float64) * float(inv_tau)
    Z = Z - Z.max(axis=1, keepdims=True)
    e = np.exp(Z)
    return e / e.sum(axis=1, keepdims=True)


def router_ref(X, Wg, inv_tau: float = 1.0) -> np.ndarray:
    """S = softmax(X Wg^T / tau) with Wg stored [E, d]."""
    return softmax_ref(widen(X) @ widen(Wg).T, inv_tau)


# ---------------------------------------------------------------------------
# Expert-choice selection (Section 2.2: T_j = TopC_i(S_ij); per routing group,
# Section 5.2: each expert chooses from the same L-token pool of its sequence)
# ---------------------------------------------------------------------------

def select_ref(S, group_offsets, capacity) -> np.ndarray:
    """sel_token[E, K_tot]: for each expert j and group g, the k_g tokens of the group
    with the largest S[:, j] (equal scores: lower token index first), listed in
    ascending token order.  Expert j's row holds group 0's tokens, then group 1's, ...
    """
    S = np.asarray(S, dtype=np.float64)
    off = np.asarray(group_offsets, dtype=np.int64)
    k = np.asarray(capacity, dtype=np.int64)
    E = S.shape[1]
    K_tot = int(k.sum())
    sel = np.empty((E, K_tot), dtype=np.int64)
    for j in range(E):
        pos = 0
        for g in range(len(k)):
            lo, hi = int(off[g]), int(off[g + 1])
            idx = np.arange(lo, hi)
            col = S[lo:hi, j]
            order = np.lexsort((idx, -col))          # score descending, index ascending
            chosen = np.sort(idx[order[: k[g]]])
            sel[j, pos: pos + k[g]] = chosen
            pos += k[g]
    return sel


def slot_ref(sel_token, n_tokens: int) -> np.ndarray:
    """slot[N, E]: row of token i in expert j's buffer, or -1 if j did not select i."""
    E, K = sel_token.shape
    slot = np.full((n_tokens, E), -1, dtype=np.int64)
    for j in range(E):
        slot[sel_token[j], j] = np.arange(K)
    return slot


def coverage_ref(sel_token, group_offsets):
    """Token drop statistic (Appendix D): experts_per_token[i] = number of experts
    whose chosen set contains token i; dropped[g] = tokens of group g that no
    expert chose (their layer output is zero)."""
    off = np.asarray(group_offsets, dtype=np.int64)
    N = int(off[-1])
    counts = np.zeros(N, dtype=np.int64)
    for row in np.asarray(sel_token):
        for i in row:
            counts[int(i)] += 1
    dropped = np.array([int(np.sum(counts[off[g]:off[g + 1]] == 0)) for g in range(len(off) - 1)],
                       dtype=np.int64)
    return counts, dropped


def bruteforce_select(col, k: int) -> tuple:
    """Among all size-k subsets, the one that no unselected entry beats under the
    order (score descending, index ascending).  Exponential; tiny inputs only."""
    col = [float(v) for v in col]
    n = len(col)
    found = []
    for sub in itertools.combinations(range(n), k):
        s = set(sub)
        ok = True
        for a in sub:
            for b in range(n):
                if b in s:
                    continue
                # b beats a if its score is higher, or equal with a lower index
                if col[b] > col[a] or (col[b] == col[a] and b < a):
                    ok = False
                    break
            if not ok:
                break
        if ok:
            found.append(sub)
    assert len(found) == 1, "the selection rule must have exactly one answer"
    return found[0]


# ---------------------------------------------------------------------------
# Experts (Appendix E: SwiGLU expert FFNs) and combine (Section 2.2)
# ---------------------------------------------------------------------------

def silu(z):
    return z / (1.0 + np.exp(-z))


def swiglu_ffn_ref(x, W1j, W3j, W2j):
    """FFN_j(x) = W2_j (SiLU(W1_j x) * (W3_j x)), rows of x are tokens."""
    x = widen(x)
    h1 = x @ widen(W1j).T
    h3 = x @ widen(W3j).T
    return (silu(h1) * h3) @ widen(W2j).T


def forward_ref(X, Wg, W1, W3, W2, group_offsets, capacity, inv_tau: float = 1.0,
                sel_token=None, shared=None, on_expert=None) -> dict:
    """Layer output y_i = sum over experts j that selected i of g_ij FFN_j(x_i),
    with g_ij = S_ij; y_i = 0 when no expert selected token i.  With shared
    experts (Ws1, Ws3, Ws2), their FFN of x_i is added to every y_i.

    If sel_token is given it replaces the selection (used to evaluate the layer on
    the selection another implementation made from its own score matrix).
    on_expert(j, O_j), if given, receives each expert's gate-weighted outputs
    O_j[r] = g_{sel[j, r], j} FFN_j(x_{sel[j, r]}) as they are computed."""
    Xf, W1f, W3f, W2f = widen(X), widen(W1), widen(W3), widen(W2)
    S = router_ref(X, Wg, inv_tau)
    sel = select_ref(S, group_offsets, capacity) if sel_token is None else np.asarray(sel_token)
    E = S.shape[1]
    Y = np.zeros_like(Xf)
    gate = np.empty(sel.shape, dtype=np.float64)
    for j in range(E):
        rows = sel[j]
        gate[j] = S[rows, j]
        o = gate[j][:, None] * swiglu_ffn_ref(Xf[rows], W1f[j], W3f[j], W2f[j])
        Y[rows] += o                               # rows are distinct within one expert
        if on_expert is not None:
            on_expert(j, o)
    if shared is not None:
        Y += shared_ffn_ref(Xf, shared)
    return {"S": S, "sel_token": sel, "gate": gate, "Y": Y}


def dense_loop_ref(X, Wg, W1, W3, W2, group_offsets, capacity, inv_tau: float = 1.0,
                   shared_experts=()):
    """The combine as an explicit loop over (expert, selected token), one vector at a
    time, plus every shared expert (a list of (W1s, W3s, W2s), one per shared
    expert) on every token.  Small inputs only."""
    Xf, W1f, W3f, W2f = widen(X), widen(W1), widen(W3), widen(W2)
    S = router_ref(X, Wg, inv_tau)
    sel = select_ref(S, group_offsets, capacity)
    Y = np.zeros_like(Xf)
    for j in range(sel.shape[0]):
        for i in sel[j]:
            x = Xf[i]
            a = silu(W1f[j] @ x) * (W3f[j] @ x)
            Y[i] = Y[i] + S[i, j] * (W2f[j] @ a)
    for (w1, w3, w2) in shared_experts:
        w1, w3, w2 = widen(w1), widen(w3), widen(w2)
        for i in range(Xf.shape[0]):
            x = Xf[i]
            Y[i] = Y[i] + w2 @ (silu(w1 @ x) * (w3 @ x))
    return Y


# ---------------------------------------------------------------------------
# Token choice (Section 2.2, the comparison policy): each token takes the
# top_k experts of its row of S (equal scores: lower expert index first) with
# gates normalised over those k experts; expert j keeps at most capacity[g] of
# the tokens of group g that chose it, the lowest token indices first, and the
# other pairs are dropped (their gate weight is lost, not renormalised).
# ---------------------------------------------------------------------------

def tc_capacity_ref(group_lengths, n_experts: int, top_k: int, cf: float):
    """Tokens each expert may keep from group g: ceil(CF k L_g / E), at most L_g;
    CF <= 0 means no cap (dropless)."""
    L = np.asarray(group_lengths, dtype=np.int64)
    if cf <= 0:
        return L.copy()
    return np.minimum(L, np.ceil(cf * top_k * L / n_experts - 1e-9).astype(np.int64))


def tc_select_ref(S, group_offsets, top_k: int, capacity):
    """Returns choice [N, top_k] (expert ids, descending score), gate [N, top_k]
    (normalised over the row's choice), kept [N, top_k] (bool) and rows, a list
    over experts of the kept tokens of each expert in ascending order."""
    S = np.asarray(S, dtype=np.float64)
    N, E = S.shape
    off = np.asarray(group_offsets, dtype=np.int64)
    choice = np.empty((N, top_k), dtype=np.int64)
    for i in range(N):
        order = np.lexsort((np.arange(E), -S[i]))     # score descending, index ascending
        choice[i] = order[:top_k]
    picked = np.take_along_axis(S, choice, 1)
    gate = picked / picked.sum(axis=1, keepdims=True)
    kept = np.zeros((N, top_k), dtype=bool)
    rows = [[] for _ in range(E)]
    for g in range(len(off) - 1):
        used = np.zeros(E, dtype=np.int64)
        for i in range(int(off[g]), int(off[g + 1])):
            for r in range(top_k):
                j = int(choice[i, r])
                if used[j] < capacity[g]:
                    used[j] += 1
                    kept[i, r] = True
                    rows[j].append(i)
    return choice, gate, kept, [np.asarray(r, dtype=np.int64) for r in rows]


def tc_forward_ref(X, Wg, W1, W3, W2, group_offsets, top_k: int, capacity,
                   inv_tau: float = 1.0, selection=None) -> dict:
    """y_i = sum over the kept pairs (i, j) of g_ij FFN_j(x_i).  selection =
    (choice, kept) replaces the selection (another implementation's, made on its
    own scores); the gates are then the normalised scores of that choice."""
    Xf = widen(X)
    S = router_ref(X, Wg, inv_tau)
    if selection is None:
        choice, gate, kept, rows = tc_select_ref(S, group_offsets, top_k, capacity)
    else:
        choice, kept = (np.asarray(a) for a in selection)
        picked = np.take_along_axis(S, choice, 1)
        gate = picked / picked.sum(axis=1, keepdims=True)
        rows = [np.asarray(sorted(int(i) for i, r in zip(*np.nonzero(kept)) if choice[i, r] == j),
                           dtype=np.int64) for j in range(S.shape[1])]
    N, E = S.shape
    G = np.zeros((N, E))
    for r in range(top_k):
        G[np.arange(N), choice[:, r]] += np.where(kept[:, r], gate[:, r], 0.0)
    Y = np.zeros_like(Xf)
    for j in range(E):
        if len(rows[j]):
            Y[rows[j]] += G[rows[j], j][:, None] * swiglu_ffn_ref(Xf[rows[j]], W1[j], W3[j], W2[j])
    return {"S": S, "choice": choice, "gate": gate, "kept": kept, "rows": rows, "G": G, "Y": Y}


def tc_forward_rows_ref(X, Wg, W1, W3, W2, choice, kept, rows, inv_tau: float = 1.0):
    """y_i of the token-choice layer for the listed tokens only, selection given."""
    rows = np.asarray(rows, dtype=np.int64)
    Xr = widen(np.asarray(X)[rows])
    S = softmax_ref(Xr @ widen(Wg).T, inv_tau)
    ch, kp = np.asarray(choice)[rows], np.asarray(kept)[rows]
    picked = np.take_along_axis(S, ch, 1)
    gate = picked / picked.sum(axis=1, keepdims=True)
    Y = np.zeros_like(Xr)
    for q in range(len(rows)):
        for r in range(ch.shape[1]):
            if kp[q, r]:
                j = int(ch[q, r])
                Y[q] += gate[q, r] * swiglu_ffn_ref(Xr[q:q + 1], W1[j], W3[j], W2[j])[0]
    return Y


# ---------------------------------------------------------------------------
# Shared experts (Appendix D: they process every token whatever the routing;
# Appendix E: 2 per MoE layer).  n_s shared SwiGLU experts of width h_s are one
# SwiGLU of width n_s h_s whose hidden units are theirs side by side
# (Ws1, Ws3 [n_s h_s, d], Ws2 [d, n_s h_s]); the output is added to the routed
# sum without a gate.
# ---------------------------------------------------------------------------

def shared_ffn_ref(X, shared):
    """FFN_shared(x) for every row x of X."""
    Ws1, Ws3, Ws2 = shared
    return swiglu_ffn_ref(X, Ws1, Ws3, Ws2)


def shared_backward_ref(X, shared, dY):
    """(dX, dWs1, dWs3, dWs2) of sum(FFN_shared(X) * dY)."""
    Ws1, Ws3, Ws2 = (widen(w) for w in shared)
    x, dy = widen(X), widen(dY)
    h1, h3 = x @ Ws1.T, x @ Ws3.T
    sg = 1.0 / (1.0 + np.exp(-h1))
    a = h1 * sg * h3
    da = dy @ Ws2
    dh3 = da * (h1 * sg)
    dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
    return dh1 @ Ws1 + dh3 @ Ws3, dh1.T @ x, dh3.T @ x, dy.T @ a


def shared_grads_units_ref(X, shared, dY, units):
    """Rows `units` of dWs1 and dWs3 and columns `units` of dWs2 (hidden units of
    the shared FFN), each needing only its own unit over all tokens."""
    Ws1, Ws3, Ws2 = shared
    u = np.asarray(units, dtype=np.int64)
    x, dy = widen(X), widen(dY)
    h1, h3 = x @ widen(np.asarray(Ws1)[u]).T, x @ widen(np.asarray(Ws3)[u]).T
    sg = 1.0 / (1.0 + np.exp(-h1))
    a = h1 * sg * h3
    da = dy @ widen(np.asarray(Ws2)[:, u])
    dh3 = da * (h1 * sg)
    dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
    return dh1.T @ x, dh3.T @ x, dy.T @ a


# ---------------------------------------------------------------------------
# Backward: exact derivatives with the selection held fixed (it is an index set)
# ---------------------------------------------------------------------------

def backward_ref(X, Wg, W1, W3, W2, dY, group_offsets, capacity, inv_tau: float = 1.0,
                 sel_token=None, shared=None, on_expert=None) -> dict:
    """Gradients of sum(Y * dY) w.r.t. X, Wg, W1, W3, W2 (and the shared experts'
    Ws1, Ws3, Ws2 when given: their FFN adds its own dX term).  The forward
    output Y comes along (the same terms), and on_expert(j, O_j) as in
    forward_ref.

    Chain, per selected pair (i, j) with x = x_i:
      O = W2_j A, A = SiLU(H1) * H3, H1 = W1_j x, H3 = W3_j x, y_i += S_ij O
      dO = S_ij dY_i,  dS_ij = <dY_i, O>
      dA = W2_j^T dO,  dW2_j += dO A^T
      dH3 = dA * SiLU(H1),  dH1 = dA * H3 * SiLU'(H1)
      dx += W1_j^T dH1 + W3_j^T dH3,  dW1_j += dH1 x^T,  dW3_j += dH3 x^T
    Router: S_i = softmax(Z_i / tau), Z = X Wg^T; dS is zero off the selection,
      dZ_i = (S_i * (dS_i - <S_i, dS_i>)) / tau,  dWg = dZ^T X,  dX += dZ Wg.
    """
    Xf, Wgf, W1f, W3f, W2f = widen(X), widen(Wg), widen(W1), widen(W3), widen(W2)
    dYf = widen(dY)
    S = router_ref(X, Wg, inv_tau)
    sel = select_ref(S, group_offsets, capacity) if sel_token is None else np.asarray(sel_token)
    E = S.shape[1]
    dX = np.zeros_like(Xf)
    dS = np.zeros_like(S)
    dW1 = np.zeros_like(W1f)
    dW3 = np.zeros_like(W3f)
    dW2 = np.zeros_like(W2f)
    Y = np.zeros_like(Xf)
    for j in range(E):
        rows = sel[j]
        x = Xf[rows]
        h1 = x @ W1f[j].T
        h3 = x @ W3f[j].T
        sg = 1.0 / (1.0 + np.exp(-h1))
        a = h1 * sg * h3
        o = a @ W2f[j].T
        g = S[rows, j]
        Y[rows] += g[:, None] * o
        if on_expert is not None:
            on_expert(j, g[:, None] * o)
        dy = dYf[rows]
        dS[rows, j] = np.sum(dy * o, axis=1)
        do = g[:, None] * dy
        da = do @ W2f[j]
        dW2[j] = do.T @ a
        dh3 = da * (h1 * sg)
        dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
        dX[rows] += dh1 @ W1f[j] + dh3 @ W3f[j]
        dW1[j] = dh1.T @ x
        dW3[j] = dh3.T @ x
    dZ = S * (dS - np.sum(S * dS, axis=1, keepdims=True)) * float(inv_tau)
    dWg = dZ.T @ Xf
    dX += dZ @ Wgf
    out = {"dX": dX, "dWg": dWg, "dW1": dW1, "dW3": dW3, "dW2": dW2, "dS": dS,
           "S": S, "sel_token": sel, "Y": Y}
    if shared is not None:
        dXs, out["dWs1"], out["dWs3"], out["dWs2"] = shared_backward_ref(Xf, shared, dYf)
        out["dX"] = dX + dXs
        out["Y"] = Y + shared_ffn_ref(Xf, shared)
    return out


def loss_ref(X, Wg, W1, W3, W2, dY, group_offsets, capacity, inv_tau, sel_token,
             shared=None) -> float:
    """sum(Y * dY) with a fixed selection: the scalar whose gradient backward_ref returns."""
    Y = forward_ref(X, Wg, W1, W3, W2, group_offsets, capacity, inv_tau, sel_token, shared)["Y"]
    return float(np.sum(Y * widen(dY)))


# ---------------------------------------------------------------------------
# Restrictions of the definitions above to a few tokens or one expert, for
# large inputs where the full evaluation is too slow in float64.  Each is
# checked against forward_ref / backward_ref on small inputs.
# ---------------------------------------------------------------------------

def forward_rows_ref(X, Wg, W1, W3, W2, sel_token, rows, inv_tau: float = 1.0,
                     shared=None) -> np.ndarray:
    """y_i for the listed tokens only, with the selection given."""
    rows = np.asarray(rows, dtype=np.int64)
    slot = slot_ref(np.asarray(sel_token), np.asarray(X).shape[0])[rows]
    Xr = widen(np.asarray(X)[rows])
    S = softmax_ref(Xr @ widen(Wg).T, inv_tau)
    Y = np.zeros_like(Xr)
    for j in range(S.shape[1]):
        q = np.nonzero(slot[:, j] >= 0)[0]          # listed tokens that expert j selected
        if len(q):
            Y[q] += S[q, j][:, None] * swiglu_ffn_ref(Xr[q], W1[j], W3[j], W2[j])
    if shared is not None:
        Y += shared_ffn_ref(Xr, shared)
    return Y


def _pair_terms(x, W1j, W3j, W2j):
    """H1, H3, sigmoid(H1), A and O for rows x of one expert."""
    h1 = x @ widen(W1j).T
    h3 = x @ widen(W3j).T
    sg = 1.0 / (1.0 + np.exp(-h1))
    a = h1 * sg * h3
    return h1, h3, sg, a, a @ widen(W2j).T


def backward_rows_ref(X, Wg, W1, W3, W2, dY, sel_token, rows, inv_tau: float = 1.0,
                      shared=None) -> np.ndarray:
    """dX_i for the listed tokens only (expert, router and shared-expert terms),
    selection given."""
    rows = np.asarray(rows, dtype=np.int64)
    slot = slot_ref(np.asarray(sel_token), np.asarray(X).shape[0])[rows]
    Xr, dYr, Wgf = widen(np.asarray(X)[rows]), widen(np.asarray(dY)[rows]), widen(Wg)
    S = softmax_ref(Xr @ Wgf.T, inv_tau)
    dX = np.zeros_like(Xr)
    dS = np.zeros_like(S)
    for j in range(S.shape[1]):
        q = np.nonzero(slot[:, j] >= 0)[0]
        if not len(q):
            continue
        h1, h3, sg, a, o = _pair_terms(Xr[q], W1[j], W3[j], W2[j])
        dS[q, j] = np.sum(dYr[q] * o, axis=1)
        da = (S[q, j][:, None] * dYr[q]) @ widen(W2[j])
        dh3 = da * (h1 * sg)
        dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
        dX[q] += dh1 @ widen(W1[j]) + dh3 @ widen(W3[j])
    dZ = S * (dS - np.sum(S * dS, axis=1, keepdims=True)) * float(inv_tau)
    if shared is not None:
        dX += shared_backward_ref(Xr, shared, dYr)[0]
    return dX + dZ @ Wgf


def expert_grads_ref(X, Wg, W1, W3, W2, dY, sel_token, j: int, inv_tau: float = 1.0):
    """(dW1_j, dW3_j, dW2_j) of one expert, selection given."""
    rows = np.asarray(sel_token)[j]
    x = widen(np.asarray(X)[rows])
    g = softmax_ref(x @ widen(Wg).T, inv_tau)[:, j]
    h1, h3, sg, a, o = _pair_terms(x, W1[j], W3[j], W2[j])
    do = g[:, None] * widen(np.asarray(dY)[rows])
    da = do @ widen(W2[j])
    dh3 = da * (h1 * sg)
    dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
    return dh1.T @ x, dh3.T @ x, do.T @ a


def expert_grads_units_ref(X, Wg, W1, W3, W2, dY, sel_token, j: int, units,
                           inv_tau: float = 1.0):
    """Rows `units` of dW1_j and dW3_j and columns `units` of dW2_j (hidden units of
    expert j), selection given: each hidden unit needs only its own pre-activations
    over the expert's rows."""
    u = np.asarray(units, dtype=np.int64)
    rows = np.asarray(sel_token)[j]
    x = widen(np.asarray(X)[rows])
    g = softmax_ref(x @ widen(Wg).T, inv_tau)[:, j]
    h1 = x @ widen(np.asarray(W1[j])[u]).T
    h3 = x @ widen(np.asarray(W3[j])[u]).T
    sg = 1.0 / (1.0 + np.exp(-h1))
    a = h1 * sg * h3
    do = g[:, None] * widen(np.asarray(dY)[rows])
    da = do @ widen(np.asarray(W2[j])[:, u])
    dh3 = da * (h1 * sg)
    dh1 = da * h3 * (sg * (1.0 + h1 * (1.0 - sg)))
    return dh1.T @ x, dh3.T @ x, do.T @ a


def router_grad_ref(X, Wg, W1, W3, W2, dY, sel_token, inv_tau: float = 1.0) -> np.ndarray:
    """dWg [E, d] with the selection given (needs every selected pair's output)."""
    Xf, dYf = widen(X), widen(dY)
    S = router_ref(X, Wg, inv_tau)
    sel = np.asarray(sel_token)
    dS = np.zeros_like(S)
    for j in range(S.shape[1]):
        rows = sel[j]
        o = _pair_terms(Xf[rows], W1[j], W3[j], W2[j])[4]
        dS[rows, j] = np.sum(dYf[rows] * o, axis=1)
    dZ = S * (dS - np.sum(S * dS, axis=1, keepdims=True)) * float(inv_tau)
    return dZ.T @ Xf
