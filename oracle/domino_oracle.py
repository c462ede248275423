"""CPU oracle for Domino's per-step drafting path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module; only the test-suite, the package smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the GPU path: it takes plain
numpy arrays (weights as fp32/fp64 values, already rounded to their storage
type by the input generator) and computes in float64 throughout, with no
activation rounding, no blocking and no fusion.

What it follows (paper sections are those of "Domino: Decoupling Causal
Modeling from Autoregressive Drafting in Speculative Decoding"):

* Sec. 4.1.1, masked-block equation: block = [anchor, MASK x (B-1)].
* Sec. 4.1.1, backbone equation: one non-autoregressive forward over the block
  conditioned on the target context.  The paper names the DFlash architecture
  without its internals; the layer used here is the Qwen3-style reading:
  pre-RMSNorm (eps 1e-6), per-head q/k RMSNorm, rotate-half RoPE (theta 1e6),
  grouped-query attention with scale 1/sqrt(d_h), SwiGLU FFN, final RMSNorm,
  no biases.  Block queries attend to every context key and to all block keys
  (no mask).  Context positions are 0..n-1, block positions n..n+B-1.
* Sec. 4.1.1, base-logit equation: L_base_i = LMHead(H_i), i = t+1..t+B-1.
* Sec. 4.1.2, causal-encoder equation: S_{i-1} = GRU(E_{<=i-1}), d_s = 1024,
  the GRU in reset-after form with input and hidden biases, gate order
  (r, z, n); initial state 0; first input the anchor's embedding.
* Sec. 4.1.2, correction equation: dL_i = W2 SiLU(W1 [H_i; S_{i-1}]) and
  L_i = L_base_i + dL_i, with r = 256 and no biases; H_i is the post-final-norm
  hidden (the LM-head input).
* Fig. 3 caption: each draft token comes from l_i + c_i and is fed back into
  the causal state (greedy: the top-1 token).
* Sec. 3.1: acceptance of the longest valid prefix plus the target's bonus
  token, tau in [1, gamma+1].
* Tie-break everywhere (top-beta, argmax, acceptance): value descending, then
  token id ascending, NaN ordered as -inf.
* Tree (the paper names tree construction without defining it): the beta
  top-ranked tokens at every depth; only the rank-0 (spine) node has children;
  breadth-first node order.

Parity pins live in tests/test_oracle_pins.py; the parts with no pin beyond the
written reading (the backbone layer wiring) are marked "parity unpinned" there.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64

from .sampling_oracle import sample_draft  # noqa: E402  (sampled drafting, Fig. 3)


# ----------------------------------------------------------------------------
# elementary operations
# ----------------------------------------------------------------------------
def rms_norm(x, gain, eps):
    """x / sqrt(mean(x^2) + eps) * gain over the last axis (Qwen3-style RMSNorm)."""
    x = np.asarray(x, F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, F64)


def rope(x, pos, theta):
    """Rotate-half rotary embedding.

    x: [rows, heads, d_h]; pos: [rows].  Pair (x_i, x_{i+d_h/2}) is rotated by
    angle pos * theta^(-2i/d_h).
    """
    x = np.asarray(x, F64)
    d = x.shape[-1]
    half = d // 2
    i = np.arange(half, dtype=F64)
    omega = np.power(F64(theta), -2.0 * i / d)
    ang = np.asarray(pos, F64)[:, None, None] * omega[None, None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s, axis=-1):
    s = np.asarray(s, F64)
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def silu(x):
    x = np.asarray(x, F64)
    return x / (1.0 + np.exp(-x))


def sigmoid(x):
    x = np.asarray(x, F64)
    return 1.0 / (1.0 + np.exp(-x))


def attention(q, k, v):
    """softmax(q k^T / sqrt(d_h)) v with grouped-query heads and no mask.

    q: [Lq, nq, d_h]; k, v: [Lk, nkv, d_h]; query head h reads kv head
    h // (nq / nkv).  Returns [Lq, nq, d_h].
    """
    q, k, v = (np.asarray(a, F64) for a in (q, k, v))
    nq, nkv, dh = q.shape[1], k.shape[1], q.shape[2]
    grp = nq // nkv
    out = np.empty_like(q)
    for h in range(nq):
        kv = h // grp
        s = q[:, h, :] @ k[:, kv, :].T / np.sqrt(F64(dh))
        out[:, h, :] = softmax(s, axis=-1) @ v[:, kv, :]
    return out


# ----------------------------------------------------------------------------
# backbone (Sec. 4.1.1)
# ----------------------------------------------------------------------------
def fuse_context(cfg, w, hidden):
    """Context features C_t (Sec. 4.1.1) from the target's hidden states.

    With cfg.ctx_fuse_layers = k > 0 a context row is the concatenation of the
    hidden states of k target layers, [n, k*d]; one linear map ctx_fc [d, k*d]
    fuses it to width d.  The paper gives the fusion no formula: this is the
    reading that the +5.3% parameter figure of Sec. 1 implies (an ~84M map at
    the Qwen3-8B shape with k = 5).  With k = 0 the rows are used as they are.
    """
    c = np.asarray(hidden, F64)
    if cfg.ctx_fuse_layers <= 0:
        return c
    return c @ np.asarray(w["ctx_fc"], F64).T


def project_context_kv(cfg, lw, hidden, positions):
    """Context K/V of one layer from target hidden states.

    K = RoPE(k_norm(W_k c)), V = W_v c at the given positions (the paper's
    context features C_t, taken into each layer through that layer's own K/V
    projections).  hidden: [n, d] -> (K, V) each [n, nkv, d_h].
    """
    nkv, dh = cfg.n_kv_heads, cfg.head_dim
    c = np.asarray(hidden, F64)
    k = (c @ np.asarray(lw["wk"], F64).T).reshape(-1, nkv, dh)
    v = (c @ np.asarray(lw["wv"], F64).T).reshape(-1, nkv, dh)
    k = rope(rms_norm(k, lw["k_norm"], cfg.rms_eps), positions, cfg.rope_theta)
    return k, v


def backbone_layer(cfg, lw, x, pos, ctx_k, ctx_v):
    """One drafter layer over the B block rows.

    x: [B, d]; pos: [B]; ctx_k, ctx_v: [n, nkv, d_h] (n may be 0).
    """
    nq, nkv, dh, eps = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps
    x = np.asarray(x, F64)
    a = rms_norm(x, lw["attn_norm"], eps)
    q = (a @ np.asarray(lw["wq"], F64).T).reshape(-1, nq, dh)
    k = (a @ np.asarray(lw["wk"], F64).T).reshape(-1, nkv, dh)
    v = (a @ np.asarray(lw["wv"], F64).T).reshape(-1, nkv, dh)
    q = rope(rms_norm(q, lw["q_norm"], eps), pos, cfg.rope_theta)
    k = rope(rms_norm(k, lw["k_norm"], eps), pos, cfg.rope_theta)
    keys = np.concatenate([np.asarray(ctx_k, F64), k], axis=0)
    vals = np.concatenate([np.asarray(ctx_v, F64), v], axis=0)
    o = attention(q, keys, vals).reshape(x.shape[0], nq * dh)
    x = x + o @ np.asarray(lw["wo"], F64).T
    y = rms_norm(x, lw["ffn_norm"], eps)
    g = y @ np.asarray(lw["w_gate"], F64).T
    u = y @ np.asarray(lw["w_up"], F64).T
    x = x + (silu(g) * u) @ np.asarray(lw["w_down"], F64).T
    return x


def masked_block(cfg, anchor):
    """[anchor, MASK, ..., MASK] of length B (Sec. 4.1.1)."""
    return np.array([int(anchor)] + [cfg.mask_id] * (cfg.block - 1), dtype=np.int64)


def draft_backbone(cfg, w, anchor, ctx_k, ctx_v, ctx_len):
    """Post-final-norm hidden states H_j for the B-1 draft positions.

    ctx_k/ctx_v: [L, max_ctx, nkv, d_h] for this batch row.  Returns [B-1, d].
    """
    n = int(ctx_len)
    x = np.asarray(np.asarray(w["embed"])[masked_block(cfg, anchor)], F64)  # rows first, then exact upcast
    pos = np.arange(n, n + cfg.block, dtype=F64)
    for l, lw in enumerate(w["layers"]):
        x = backbone_layer(cfg, lw, x, pos, ctx_k[l, :n], ctx_v[l, :n])
    h = rms_norm(x, w["final_norm"], cfg.rms_eps)
    return h[1:]


def base_logits(w, h):
    """L_base = LMHead(H) for the draft positions: [B-1, V]."""
    return np.asarray(h, F64) @ np.asarray(w["lm_head"], F64).T


# ----------------------------------------------------------------------------
# Domino head (Sec. 4.1.2, Fig. 3)
# ----------------------------------------------------------------------------
def gru_cell(w, e, h):
    """One GRU step, reset-after form, gates ordered (r, z, n)."""
    ds = np.asarray(h).shape[-1]
    gi = np.asarray(w["gru_w_ih"], F64) @ np.asarray(e, F64) + np.asarray(w["gru_b_ih"], F64)
    gh = np.asarray(w["gru_w_hh"], F64) @ np.asarray(h, F64) + np.asarray(w["gru_b_hh"], F64)
    r = sigmoid(gi[:ds] + gh[:ds])
    z = sigmoid(gi[ds:2 * ds] + gh[ds:2 * ds])
    c = np.tanh(gi[2 * ds:] + r * gh[2 * ds:])
    return (1.0 - z) * c + z * np.asarray(h, F64)


def correction(w, h_j, s):
    """dL = W2 SiLU(W1 [H_j; S])."""
    hs = np.concatenate([np.asarray(h_j, F64), np.asarray(s, F64)])
    u = silu(np.asarray(w["w1"], F64) @ hs)
    return np.asarray(w["w2"], F64) @ u


def order_key(vals):
    """Values with NaN mapped to -inf (the ordering used for every selection)."""
    v = np.array(vals, dtype=F64, copy=True)
    v[np.isnan(v)] = -np.inf
    return v


def top_beta(vals, beta):
    """First beta token ids under (value desc, id asc); returns (ids, values).

    A sort of the whole vocabulary, by definition of the order.
    """
    v = order_key(vals)
    ids = np.arange(v.shape[0])
    order = np.lexsort((ids, -v))
    sel = order[:beta]
    return sel.astype(np.int32), np.asarray(vals, F64)[sel]


def argmax_total(vals):
    """Smallest id among the maximal values, NaN as -inf."""
    v = order_key(vals)
    m = np.max(v)
    return int(np.flatnonzero(v == m)[0])


def domino_head(cfg, w, h, lbase, anchor, beta, forced=None, sampling=None, gaps_out=None):
    """Sequential rollout over the B-1 draft positions for one batch row.

    Returns (topk_ids [B-1, beta], topk_vals [B-1, beta], final logits
    [B-1, V], causal states [B-1, d_s], drafted tokens [B-1]).

    sampling = (temperature, seed, row): each position's token is drawn from
    softmax(final / T) (sampling_oracle.sample_draft; beta must be 1) and
    topk_vals holds its final logit; the draw's key gap is appended to gaps_out.
    Teacher forcing (forced) still decides the fed-back tokens.
    """
    depth = cfg.block - 1
    s = np.zeros(cfg.gru_hidden, F64)
    y = int(anchor)
    embed = w["embed"]
    ids = np.empty((depth, beta), np.int32)
    vals = np.empty((depth, beta), F64)
    final = np.empty((depth, np.asarray(lbase).shape[1]), F64)
    states = np.empty((depth, cfg.gru_hidden), F64)
    drafted = np.empty(depth, np.int32)
    for j in range(depth):
        s = gru_cell(w, np.asarray(embed[y], F64), s)          # S_{j-1} sees y_0..y_{j-1}
        states[j] = s
        final[j] = np.asarray(lbase[j], F64) + correction(w, h[j], s)
        if sampling is None:
            ids[j], vals[j] = top_beta(final[j], beta)
        else:
            assert beta == 1, "sampled drafting is defined for one token per position"
            temperature, seed, row = sampling
            tok, gap = sample_draft(final[j], temperature, seed, row, j + 1)
            ids[j, 0], vals[j, 0] = tok, final[j][tok]
            if gaps_out is not None:
                gaps_out.append(gap)
        y = int(forced[j]) if forced is not None else int(ids[j, 0])
        drafted[j] = y
    return ids, vals, final, states, drafted


# ----------------------------------------------------------------------------
# one draft step for a batch
# ----------------------------------------------------------------------------
def draft_step(cfg, w, anchor, ctx_lens, ctx_k, ctx_v, beta, forced=None,
               ctx_hidden=None, sampling=None, rows=None):
    """Full draft step.

    anchor, ctx_lens: [bs]; ctx_k/ctx_v: [L, bs, max_ctx, nkv, d_h]; forced:
    optional [bs, B-1]; ctx_hidden: optional [bs, n_new, cfg.ctx_width] target
    hidden states, fused (fuse_context) and projected into positions
    [ctx_len - n_new, ctx_len) of every layer before drafting.
    sampling: optional (temperature, seed) for sampled drafting; `rows` gives
    the batch-row index each row's random streams use (default 0..bs-1).
    Returns a dict of arrays with a leading batch axis ("sample_gap" [bs, B-1]
    when sampling).
    """
    bs = len(anchor)
    ctx_k = np.array(ctx_k, dtype=F64, copy=True)
    ctx_v = np.array(ctx_v, dtype=F64, copy=True)
    out = {k: [] for k in ("topk_ids", "topk_vals", "base_logits", "final_logits",
                           "hidden", "states", "drafted")}
    for b in range(bs):
        n = int(ctx_lens[b])
        if ctx_hidden is not None and ctx_hidden.shape[1] > 0:
            n_new = ctx_hidden.shape[1]
            pos = np.arange(n - n_new, n, dtype=F64)
            c = fuse_context(cfg, w, ctx_hidden[b])
            for l, lw in enumerate(w["layers"]):
                k, v = project_context_kv(cfg, lw, c, pos)
                ctx_k[l, b, n - n_new:n] = k
                ctx_v[l, b, n - n_new:n] = v
        h = draft_backbone(cfg, w, anchor[b], ctx_k[:, b], ctx_v[:, b], n)
        lb = base_logits(w, h)
        gaps = []
        smp = None if sampling is None else (sampling[0], sampling[1], b if rows is None else int(rows[b]))
        ids, vals, final, states, drafted = domino_head(
            cfg, w, h, lb, anchor[b], beta, None if forced is None else forced[b], smp, gaps)
        for k, v in zip(out, (ids, vals, lb, final, h, states, drafted)):
            out[k].append(v)
        if sampling is not None:
            out.setdefault("sample_gap", []).append(np.array(gaps))
    res = {k: np.stack(v) for k, v in out.items()}
    res["ctx_k"], res["ctx_v"] = ctx_k, ctx_v
    return res


# ----------------------------------------------------------------------------
# draft tree and greedy acceptance (Sec. 3.1)
# ----------------------------------------------------------------------------
def build_tree(topk_ids, anchor, ctx_lens):
    """Spine-and-leaves draft tree in breadth-first order.

    Node 0 is the anchor (parent -1, depth 0, position n).  Node
    1 + (d-1)*beta + rho holds the rank-rho token of depth d, at depth d and
    position n + d; its parent is the root for d = 1 and the spine node of
    depth d-1 otherwise.  mask[i][k] = 1 iff k is i or an ancestor of i.
    """
    topk_ids = np.asarray(topk_ids)
    bs, depth, beta = topk_ids.shape
    nn = 1 + depth * beta
    tok = np.empty((bs, nn), np.int32)
    par = np.empty((bs, nn), np.int32)
    dep = np.empty((bs, nn), np.int32)
    pos = np.empty((bs, nn), np.int32)
    mask = np.zeros((bs, nn, nn), np.uint8)
    for b in range(bs):
        n = int(ctx_lens[b])
        tok[b, 0], par[b, 0], dep[b, 0], pos[b, 0] = int(anchor[b]), -1, 0, n
        for d in range(1, depth + 1):
            for rho in range(beta):
                i = 1 + (d - 1) * beta + rho
                tok[b, i] = topk_ids[b, d - 1, rho]
                par[b, i] = 0 if d == 1 else 1 + (d - 2) * beta
                dep[b, i] = d
                pos[b, i] = n + d
        for i in range(nn):
            k = i
            while k >= 0:
                mask[b, i, k] = 1
                k = par[b, k]
    return {"node_token": tok, "node_parent": par, "node_depth": dep,
            "node_pos": pos, "ancestor_mask": mask}


def verify_accept(node_token, node_parent, target_logits, block=16):
    """Greedy acceptance: walk from the root while a child's token equals the
    target's argmax at the current node; the argmax at the last accepted node is
    the bonus token.

    Returns accept_len [bs] (tau - 1), accepted_nodes [bs, B-1] (-1 padded),
    out_tokens [bs, B] (accepted tokens then the bonus, -1 padded).
    """
    node_token = np.asarray(node_token)
    node_parent = np.asarray(node_parent)
    bs, nn = node_token.shape
    acc_len = np.zeros(bs, np.int32)
    acc_nodes = np.full((bs, block - 1), -1, np.int32)
    out_tok = np.full((bs, block), -1, np.int32)
    for b in range(bs):
        cur, a = 0, 0
        while True:
            r = argmax_total(target_logits[b, cur])
            nxt = -1
            for c in range(nn):
                if node_parent[b, c] == cur and node_token[b, c] == r:
                    nxt = c
                    break
            if nxt < 0:
                break
            acc_nodes[b, a] = nxt
            out_tok[b, a] = node_token[b, nxt]
            a += 1
            cur = nxt
        acc_len[b] = a
        out_tok[b, a] = argmax_total(target_logits[b, cur])
    return {"accept_len": acc_len, "accepted_nodes": acc_nodes, "out_tokens": out_tok}


def as_f64_weights(w, keep=()):
    """Copy a weight dict to float64 once, so repeated oracle calls do not convert.

    Entries named in `keep` stay as they are (e.g. the embedding table, of which
    only a few rows are ever read; the rows are upcast exactly where used)."""
    out = {}
    for k, v in w.items():
        if k == "layers":
            out[k] = [{kk: np.asarray(vv, F64) for kk, vv in lw.items()} for lw in v]
        elif k in keep:
            out[k] = v
        else:
            out[k] = np.asarray(v, F64)
    return out
