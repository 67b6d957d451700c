"""CPU oracle for the EC2MoE hot path: the group-gated MoE layer forward and the
low-rank encoder/decoder at the end-cloud cut.

TEST INFRASTRUCTURE, NOT PRODUCT CODE. Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import or run this module. The HIP library
never calls it, and it shares no code with the HIP library: it reads plain NumPy
arrays (the exact values of the inputs, upcast to float64) and computes every step
in float64 with no blocking, fusion or reordering beyond what the definitions say.

Sources (EC2MoE, arXiv 2508.06024):
  * Mixture-of-Experts, Eq. (1): y = sum_i G(x)_i E_i(x) with sum_i G(x)_i = 1.
  * Local Expert Selection, Eq. (4): the candidate set E_local; here a bitmask.
  * Lightweight Group Gate Network, Eq. (5): per-group softmax gate over the
    group's M_k experts; Eq. (6): the global softmax over the K groups
    (stage 1); Eq. (7): the fused probability g_i = p_group^(k) * p_local,i^(k).
  * Encoder-Decoder based on Low-Rank Compression: Z = U^T X V at the end,
    X_hat = U_hat Z V_hat^T in the cloud.
  * Parameter Selection: top-1 routing in the paper's runs; top-k in general.
  * Eq. (8): the codec's reconstruction loss; with lambda = 0 (no task loss) its
    minimiser for one slice is the truncated SVD (codec_fit_hosvd).

Readings where the paper is silent (each is also listed with the design notes):
  * the candidate filter acts before both softmaxes: non-candidates get no
    probability and a group without candidates drops out of the group softmax;
  * experts are grouped contiguously: group k holds experts [k*M/K, (k+1)*M/K), or
    groups of given sizes M_k in order (Eq. 5 allows unequal groups);
  * group-focused evaluation (the closing remark of HL-GGN) as an option: per token only
    the top-G groups by p_group keep their experts (ties to the lower group index), more
    groups in the same order while the kept ones hold fewer than k candidates; p_group
    stays the softmax over all groups with a candidate;
  * top-k orders by descending g, exact ties going to the lower expert index;
    the selected weights are renormalised to sum to 1 (Eq. (1)'s constraint
    applied to the sparse gate) unless renormalize=False;
  * the expert network is a SwiGLU feed-forward layer without biases:
    E(x) = W_down (silu(W_gate x) * (W_up x)), silu(z) = z / (1 + exp(-z));
    or, for the paper's own setting (a Switch Transformer base model,
    Experimental Setup), a two-layer ReLU feed-forward layer without biases:
    E(x) = W_down relu(W_in x);
  * tokens are permuted into per-expert segments by a stable sort on the expert
    id of each (token, slot) assignment a = t*k + j;
  * the codec acts on the [T][d] block of hidden states (h = tokens, w = model
    width, one slice), and U_hat, V_hat are inputs of their own; with c slices
    (X in R^{h x w x c}, one slice per sequence of a batch) every slice
    X[s] = rows s*h .. (s+1)*h - 1 is coded with the same U, V.
"""
from __future__ import annotations

import numpy as np


class TooFewCandidates(ValueError):
    """The candidate set holds fewer experts than the top-k asks for."""


# ----------------------------------------------------------------------------- Eq. (4)

def candidate_set(mask_words, n_experts):
    """Experts whose bit is set in the candidate mask (bit e of word e // 64)."""
    return [e for e in range(n_experts) if (int(mask_words[e // 64]) >> (e % 64)) & 1]


def expert_groups(n_experts, n_groups, group_sizes=None):
    """Contiguous groups: equal, group k = experts [k*M/K, (k+1)*M/K), or of the given
    sizes M_k (Eq. 5: M = sum_k M_k), group k starting after groups 0..k-1."""
    if group_sizes is None:
        if n_experts % n_groups:
            raise ValueError("the number of groups must divide the number of experts")
        group_sizes = [n_experts // n_groups] * n_groups
    group_sizes = [int(m) for m in group_sizes]
    if len(group_sizes) != n_groups or min(group_sizes) < 1 or sum(group_sizes) != n_experts:
        raise ValueError("group sizes must be K positive counts summing to M")
    starts = np.concatenate([[0], np.cumsum(group_sizes)])
    return [list(range(int(starts[k]), int(starts[k + 1]))) for k in range(n_groups)]


def softmax(v):
    """Softmax of a 1-D float64 vector."""
    v = np.asarray(v, dtype=np.float64)
    e = np.exp(v - v.max())
    return e / e.sum()


# ----------------------------------------------------------------------------- Eq. (5)-(7)

def _token_gate(group_logits_t, local_logits_t, cand_in_group, active, top_groups, min_candidates):
    """Eq. 5-7 for one token: (p_group over the active groups, {expert: g} of the kept groups).

    top_groups = G > 0 (group-focused evaluation, HL-GGN): only the groups ranked first by
    p_group (ties to the lower group index) keep their experts; groups are kept in that order
    until G are kept and together they hold at least min_candidates candidates. p_group is
    the softmax over all active groups either way."""
    p_group = softmax(group_logits_t[active])
    kept = list(active)
    if top_groups and top_groups < len(active):
        order = sorted(range(len(active)), key=lambda a: (-p_group[a], active[a]))
        kept, held = [], 0
        for a in order:
            if len(kept) >= top_groups and held >= min_candidates:
                break
            kept.append(active[a])
            held += len(cand_in_group[active[a]])
    g = {}
    for a, k in enumerate(active):
        if k not in kept:
            continue
        members = cand_in_group[k]
        p_local = softmax(local_logits_t[members])
        for i, pl in zip(members, p_local):
            g[i] = p_group[a] * pl
    return g


def _gate_all(x, w_global, b_global, w_local, b_local, mask_words, n_groups, group_sizes,
              top_groups, min_candidates):
    """(g [T][M], per token the sorted candidates of its kept groups)."""
    x = np.asarray(x, dtype=np.float64)
    T = x.shape[0]
    M = w_local.shape[0]
    local_logits = x @ np.asarray(w_local, np.float64).T + np.asarray(b_local, np.float64)
    group_logits = x @ np.asarray(w_global, np.float64).T + np.asarray(b_global, np.float64)
    cand = set(candidate_set(mask_words, M))
    groups = expert_groups(M, n_groups, group_sizes)
    cand_in_group = [[i for i in grp if i in cand] for grp in groups]
    active = [k for k in range(n_groups) if cand_in_group[k]]

    g = np.zeros((T, M), dtype=np.float64)
    kept = []
    for t in range(T):
        gt = _token_gate(group_logits[t], local_logits[t], cand_in_group, active, top_groups, min_candidates)
        for i, v in gt.items():
            g[t, i] = v
        kept.append(sorted(gt))
    return g, kept


def group_gate_probs(x, w_global, b_global, w_local, b_local, mask_words, n_groups,
                     group_sizes=None, top_groups=0, min_candidates=1):
    """Fused expert distribution g [T][M] of the lightweight group gate.

    Stage 1 (Eq. 6): p_group = Softmax(W_global x + b_global) over the groups that
    hold at least one candidate. Stage 2 (Eq. 5): inside group k,
    p_local^(k) = Softmax(W_k x + b_k) over the group's candidates. Fusion (Eq. 7):
    g_i = p_group^(k) * p_local,i^(k). Non-candidates get g = 0, and so do the experts of
    groups left out by top_groups (see _token_gate).
    """
    return _gate_all(x, w_global, b_global, w_local, b_local, mask_words, n_groups, group_sizes,
                     top_groups, min_candidates)[0]


def topk_select(g_row, cand, k):
    """The k candidates with the largest g, in descending order; ties -> lower index."""
    cand = sorted(cand)
    if len(cand) < k:
        raise TooFewCandidates(f"{len(cand)} candidates for top-{k}")
    order = sorted(cand, key=lambda i: (-g_row[i], i))
    return order[:k]


def group_gate(x, w_global, b_global, w_local, b_local, mask_words, n_groups, top_k,
               renormalize=True, group_sizes=None, top_groups=0):
    """Routing of every token: (idx int32 [T][k], w float64 [T][k], g float64 [T][M]).

    w holds g of the selected experts, divided by their sum when renormalize is set. With
    top_groups = G > 0 the top-k is taken among the candidates of the kept groups only.
    """
    M = w_local.shape[0]
    cand = candidate_set(mask_words, M)
    if len(cand) < top_k:
        raise TooFewCandidates(f"{len(cand)} candidates for top-{top_k}")
    g, kept = _gate_all(x, w_global, b_global, w_local, b_local, mask_words, n_groups, group_sizes,
                        top_groups, top_k)
    T = g.shape[0]
    idx = np.zeros((T, top_k), dtype=np.int32)
    w = np.zeros((T, top_k), dtype=np.float64)
    for t in range(T):
        sel = topk_select(g[t], kept[t], top_k)
        idx[t] = sel
        w[t] = g[t, sel]
        if renormalize:
            w[t] = w[t] / w[t].sum()
    return idx, w, g


# ----------------------------------------------------------------------------- dispatch

def permute(idx, n_experts):
    """Per-expert segments of the (token, slot) assignments a = t*k + j.

    Returns seg_offsets [M+1] (segment e = positions [seg[e], seg[e+1])),
    perm_src [T*k] (token of each position) and inv_perm [T*k] (position of each
    assignment). Within a segment the assignments keep ascending order.
    """
    idx = np.asarray(idx)
    k = idx.shape[1]
    flat = idx.reshape(-1).astype(np.int64)
    order = np.argsort(flat, kind="stable")
    seg = np.zeros(n_experts + 1, dtype=np.int64)
    seg[1:] = np.cumsum(np.bincount(flat, minlength=n_experts))
    perm_src = (order // k).astype(np.int32)
    inv_perm = np.empty(flat.size, dtype=np.int32)
    inv_perm[order] = np.arange(flat.size, dtype=np.int32)
    return seg.astype(np.int32), perm_src, inv_perm


# ----------------------------------------------------------------------------- experts, Eq. (1)

def silu(z):
    return z / (1.0 + np.exp(-z))


def swiglu_expert(x_rows, w_gate_up_e, w_down_e):
    """E(x) = W_down (silu(W_gate x) * (W_up x)) for a block of rows."""
    H = w_down_e.shape[1]
    h = np.asarray(x_rows, np.float64) @ np.asarray(w_gate_up_e, np.float64).T
    act = silu(h[:, :H]) * h[:, H:]
    return act @ np.asarray(w_down_e, np.float64).T


def relu_expert(x_rows, w_in_e, w_down_e):
    """E(x) = W_down relu(W_in x) for a block of rows (the Switch Transformer FFN)."""
    h = np.asarray(x_rows, np.float64) @ np.asarray(w_in_e, np.float64).T
    return np.maximum(h, 0.0) @ np.asarray(w_down_e, np.float64).T


EXPERTS = {"swiglu": swiglu_expert, "relu": relu_expert}


def expert_outputs(x, idx, w_gate_up, w_down, activation="swiglu"):
    """Y_perm [T*k][d]: every assignment's expert output, in segment order.
    w_gate_up[e] / w_down[e] may be any per-expert indexable of 2-D arrays; for ReLU
    experts w_gate_up[e] is W_in [H][d]."""
    expert = EXPERTS[activation]
    M = len(w_gate_up)
    seg, perm_src, inv_perm = permute(idx, M)
    x = np.asarray(x, np.float64)
    d = x.shape[1]
    y_perm = np.zeros((perm_src.size, d), dtype=np.float64)
    for e in range(M):
        lo, hi = int(seg[e]), int(seg[e + 1])
        if hi > lo:
            y_perm[lo:hi] = expert(x[perm_src[lo:hi]], w_gate_up[e], w_down[e])
    return y_perm, seg, perm_src, inv_perm


def combine(y_perm, inv_perm, w):
    """Eq. (1): y[t] = sum_j w[t, j] * E_{idx[t,j]}(x_t), summed over slots j in order."""
    w = np.asarray(w, np.float64)
    T, k = w.shape
    y = np.zeros((T, y_perm.shape[1]), dtype=np.float64)
    for j in range(k):
        y += w[:, j:j + 1] * y_perm[inv_perm.reshape(T, k)[:, j]]
    return y


def moe_forward(x, idx, w, w_gate_up, w_down, activation="swiglu"):
    """The sparse MoE output y [T][d] for given routing (idx, w)."""
    y_perm, _, _, inv_perm = expert_outputs(x, idx, w_gate_up, w_down, activation)
    return combine(y_perm, inv_perm, w)


# ----------------------------------------------------------------------------- codec

def lowrank_encode(x, u, v):
    """Z = U^T X V."""
    return np.asarray(u, np.float64).T @ np.asarray(x, np.float64) @ np.asarray(v, np.float64)


def lowrank_decode(z, u_hat, v_hat):
    """X_hat = U_hat Z V_hat^T."""
    return np.asarray(u_hat, np.float64) @ np.asarray(z, np.float64) @ np.asarray(v_hat, np.float64).T


# ----------------------------------------------------------------------------- the layer

def layer(x, mask_words, w_global, b_global, w_local, b_local, w_gate_up, w_down,
          u, v, u_hat, v_hat, n_groups, top_k, renormalize=True, activation="swiglu",
          codec_slices=1, top_groups=0):
    """Routing is taken on the end side from X; the experts run in the cloud on the
    reconstruction X_hat = decode(encode(X)), slice by slice. Returns a dict of every
    stage output (z is [r_h][r_w] for one slice, [c][r_h][r_w] for c > 1)."""
    idx, w, g = group_gate(x, w_global, b_global, w_local, b_local, mask_words,
                           n_groups, top_k, renormalize, top_groups=top_groups)
    x = np.asarray(x, np.float64)
    h = x.shape[0] // codec_slices
    zs = [lowrank_encode(x[s * h:(s + 1) * h], u, v) for s in range(codec_slices)]
    x_hat = np.concatenate([lowrank_decode(z_s, u_hat, v_hat) for z_s in zs], axis=0)
    z = zs[0] if codec_slices == 1 else np.stack(zs)
    y = moe_forward(x_hat, idx, w, w_gate_up, w_down, activation)
    return {"idx": idx, "w": w, "g": g, "z": z, "x_hat": x_hat, "y": y}


# ----------------------------------------------------------------------------- codec fitting, Eq. (8) with lambda = 0

def _unfold_rows(xs):
    """Mode-1 unfolding [X_1 X_2 ... X_c] (h x c*w) of slices xs [c][h][w]."""
    xs = np.asarray(xs, np.float64)
    return np.concatenate(list(xs), axis=1)


def _unfold_cols(xs):
    """Mode-2 unfolding [X_1^T X_2^T ... X_c^T] (w x c*h)."""
    xs = np.asarray(xs, np.float64)
    return np.concatenate([x.T for x in xs], axis=1)


def codec_fit_hosvd(xs, r_h, r_w):
    """Data-free fit of the codec projections (Eq. 8 with lambda = 0): U = the r_h leading left
    singular vectors of the mode-1 unfolding of the calibration slices, V = the r_w leading
    left singular vectors of the mode-2 unfolding (the truncated higher-order SVD). For one
    slice this is the truncated SVD of X, the minimiser of ||X - U U^T X V V^T||^2
    (Eckart-Young)."""
    u = np.linalg.svd(_unfold_rows(xs), full_matrices=False)[0][:, :r_h]
    v = np.linalg.svd(_unfold_cols(xs), full_matrices=False)[0][:, :r_w]
    return u, v


def orthonormal_basis(y):
    """Q of the QR factorisation y = Q R with R's diagonal positive (unique for full column rank)."""
    q, r = np.linalg.qr(np.asarray(y, np.float64))
    s = np.sign(np.diag(r))
    s[s == 0] = 1.0
    return q * s


def codec_fit_subspace(xs, omega_u, omega_v, iters):
    """The same projections by subspace iteration on the Gram matrices (Halko, Martinsson and
    Tropp, 2011, Alg. 4.4 applied to a symmetric matrix): A = sum_s X_s X_s^T, B = sum_s X_s^T X_s;
    Q_0 = orth(Omega), Q_i = orth(A Q_{i-1}) (resp. B) for i = 1..iters; U = Q_iters for A, V for B.
    The returned bases span the leading subspaces once iters is large enough for the spectral gap;
    the projector U U^T does not depend on the basis chosen inside the subspace."""
    xs = np.asarray(xs, np.float64)
    a = sum(x @ x.T for x in xs)
    b = sum(x.T @ x for x in xs)

    def iterate(g, omega):
        q = orthonormal_basis(omega)
        for _ in range(iters):
            q = orthonormal_basis(g @ q)
        return q

    return iterate(a, omega_u), iterate(b, omega_v)
