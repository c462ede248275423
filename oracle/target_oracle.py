"""CPU oracle for the target model's tree-verify forward and the cache commit.

TEST INFRASTRUCTURE ONLY (same rules as domino_oracle: only the tests, the
package smoke check and the benchmark's CPU-baseline leg use it; it shares no
code with the GPU path).  Float64 throughout; weights may be passed in their
fp32 storage values (each matrix is upcast exactly where it is used).

What it follows:
* Sec. 3.1: the target model scores every drafted candidate in one forward pass
  and the longest valid prefix is accepted (then domino_oracle.verify_accept).
  The candidates form the draft tree of domino_oracle.build_tree: node i holds
  a token at position node_pos[i]; node 0 is the anchor.
* The targets of the workloads are Qwen3 decoders: the same layer as the
  drafter's reading (pre-RMSNorm, per-head q/k RMSNorm, rotate-half RoPE,
  grouped-query attention, SwiGLU, final RMSNorm, no biases), with the target's
  own depth.  The paper gives no internals; parity is unpinned beyond this
  written rule, as for the drafter's layers.
* Tree attention (reading; the paper names the verification pass only): node i
  attends to every cached context position and to the nodes k with
  ancestor_mask[i][k] = 1 (itself and its ancestors), so each node sees exactly
  the sequence of its root-to-node path, as plain causal decoding would.
* Cache commit (reading): the anchor is the previous cycle's bonus token and has
  no cached K/V yet (context 0..n-1, anchor at n).  After acceptance of a path
  of a nodes, the cache grows by the K/V of node 0 and of the accepted nodes at
  positions n, n+1, ..., n+a; the new context length is n + 1 + a and the bonus
  token becomes the next anchor.
"""
from __future__ import annotations

import numpy as np

from .domino_oracle import rms_norm, rope, silu, softmax

F64 = np.float64


def masked_attention(q, k, v, allow):
    """softmax(q k^T / sqrt(d_h), over allowed keys only) v, grouped-query heads.

    q: [Lq, nq, d_h]; k, v: [Lk, nkv, d_h]; allow: [Lq, Lk] bool (every row
    allows at least one key).  Query head h reads kv head h // (nq / nkv).
    """
    q, k, v = (np.asarray(a, F64) for a in (q, k, v))
    allow = np.asarray(allow, bool)
    nq, nkv, dh = q.shape[1], k.shape[1], q.shape[2]
    grp = nq // nkv
    out = np.empty_like(q)
    for h in range(nq):
        kv = h // grp
        s = q[:, h, :] @ k[:, kv, :].T / np.sqrt(F64(dh))
        s = np.where(allow, s, -np.inf)
        out[:, h, :] = softmax(s, axis=-1) @ v[:, kv, :]
    return out


def target_layer(cfg, lw, x, pos, ctx_k, ctx_v, tree_mask):
    """One target layer over the N+1 tree nodes of one batch row.

    x: [N+1, d]; pos: [N+1]; ctx_k, ctx_v: [n, nkv, d_h]; tree_mask [N+1, N+1].
    Returns (x, k, v) with the nodes' post-RoPE keys and values [N+1, nkv, d_h].
    """
    nq, nkv, dh, eps = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps
    x = np.asarray(x, F64)
    a = rms_norm(x, lw["attn_norm"], eps)
    q = (a @ np.asarray(lw["wq"], F64).T).reshape(-1, nq, dh)
    k = (a @ np.asarray(lw["wk"], F64).T).reshape(-1, nkv, dh)
    v = (a @ np.asarray(lw["wv"], F64).T).reshape(-1, nkv, dh)
    q = rope(rms_norm(q, lw["q_norm"], eps), pos, cfg.rope_theta)
    k = rope(rms_norm(k, lw["k_norm"], eps), pos, cfg.rope_theta)
    n = np.asarray(ctx_k).shape[0]
    keys = np.concatenate([np.asarray(ctx_k, F64), k], axis=0)
    vals = np.concatenate([np.asarray(ctx_v, F64), v], axis=0)
    allow = np.concatenate([np.ones((x.shape[0], n), bool), np.asarray(tree_mask, bool)], axis=1)
    o = masked_attention(q, keys, vals, allow).reshape(x.shape[0], nq * dh)
    x = x + o @ np.asarray(lw["wo"], F64).T
    y = rms_norm(x, lw["ffn_norm"], eps)
    g = y @ np.asarray(lw["w_gate"], F64).T
    u = y @ np.asarray(lw["w_up"], F64).T
    x = x + (silu(g) * u) @ np.asarray(lw["w_down"], F64).T
    return x, k, v


def verify_forward(cfg, w, node_token, node_pos, ancestor_mask, ctx_lens, ctx_k, ctx_v):
    """Target logits of every tree node.

    node_token, node_pos: [bs, N+1]; ancestor_mask: [bs, N+1, N+1];
    ctx_k, ctx_v: [L, bs, max_ctx, nkv, d_h].  Returns a dict with
    logits [bs, N+1, V] and the nodes' keys/values node_k, node_v
    [L, bs, N+1, nkv, d_h].
    """
    node_token = np.asarray(node_token)
    bs, nn = node_token.shape
    L = len(w["layers"])
    logits = []
    node_k = np.empty((L, bs, nn, cfg.n_kv_heads, cfg.head_dim))
    node_v = np.empty_like(node_k)
    for b in range(bs):
        n = int(ctx_lens[b])
        x = np.asarray(np.asarray(w["embed"])[node_token[b].astype(np.int64)], F64)
        pos = np.asarray(node_pos[b], F64)
        for l, lw in enumerate(w["layers"]):
            x, k, v = target_layer(cfg, lw, x, pos, ctx_k[l, b, :n], ctx_v[l, b, :n], ancestor_mask[b])
            node_k[l, b], node_v[l, b] = k, v
        h = rms_norm(x, w["final_norm"], cfg.rms_eps)
        logits.append(h @ np.asarray(w["lm_head"], F64).T)
    return {"logits": np.stack(logits), "node_k": node_k, "node_v": node_v}


def commit(ctx_k, ctx_v, ctx_lens, node_k, node_v, accept_len, accepted_nodes):
    """Cache after acceptance: node 0 at position n, the accepted node of depth
    d at position n + d.  Returns (ctx_k, ctx_v, new_ctx_lens) as new float64 arrays."""
    ctx_k = np.array(ctx_k, dtype=F64, copy=True)
    ctx_v = np.array(ctx_v, dtype=F64, copy=True)
    bs = len(ctx_lens)
    new_lens = np.empty(bs, np.int32)
    for b in range(bs):
        n, a = int(ctx_lens[b]), int(accept_len[b])
        path = [0] + [int(accepted_nodes[b][d]) for d in range(a)]
        for d, node in enumerate(path):
            ctx_k[:, b, n + d] = node_k[:, b, node]
            ctx_v[:, b, n + d] = node_v[:, b, node]
        new_lens[b] = n + 1 + a
    return ctx_k, ctx_v, new_lens
