"""Pins for the target-verify oracle (tree-attention forward and cache commit),
on the CPU: torch's attention with an explicit mask, agreement of one tree
forward with token-by-token causal decoding through the commit, agreement of
a leaf with the chain that substitutes it, and a closed form with the
attention and FFN outputs switched off."""
import numpy as np
import pytest

import oracle
import synth

tg = oracle.target_oracle
F64 = np.float64


def _tiny(layers=2, **kw):
    cfg = synth.get_config("tiny_target").with_(n_layers=layers, **kw)
    w = synth.make_target_weights(cfg, seed=7, gain_std=0.1)
    return cfg, w


def _ctx(cfg, n, max_ctx, seed=7):
    inp = synth.make_inputs(cfg.with_(batch=1, ctx=n), seed=seed, max_ctx=max_ctx)
    return inp["ctx_k"], inp["ctx_v"]


def _chain(tokens, n):
    """A chain tree: node i holds tokens[i] at position n + i; ancestors are 0..i."""
    m = len(tokens)
    return (np.asarray(tokens, np.int32)[None], (n + np.arange(m, dtype=np.int32))[None],
            np.tril(np.ones((m, m), np.uint8))[None])


def test_masked_attention_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    q = rng.normal(size=(7, 4, 16))
    k = rng.normal(size=(11, 2, 16))
    v = rng.normal(size=(11, 2, 16))
    allow = rng.random((7, 11)) < 0.5
    allow[np.arange(7), np.arange(7) + 4] = True      # every row keeps a key
    got = tg.masked_attention(q, k, v, allow)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).repeat_interleave(2, dim=1).permute(1, 0, 2)
    tv = torch.from_numpy(v).repeat_interleave(2, dim=1).permute(1, 0, 2)
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(allow))
    np.testing.assert_allclose(got, want.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_chain_forward_equals_token_by_token_decoding():
    """One forward over a chain gives, at every node, the logits that decoding
    the tokens one at a time (each a one-node tree, committed into the cache
    before the next) gives."""
    cfg, w = _tiny()
    n, m, mc = 20, 6, 64
    ck, cv = _ctx(cfg, n, mc)
    toks = np.random.default_rng(1).integers(0, cfg.vocab, size=m)
    tok, pos, mask = _chain(toks, n)
    full = tg.verify_forward(cfg, w, tok, pos, mask, [n], ck, cv)
    lens = np.array([n], np.int32)
    for i in range(m):
        one = tg.verify_forward(cfg, w, tok[:, i:i + 1], pos[:, i:i + 1], np.ones((1, 1, 1), np.uint8), lens, ck, cv)
        np.testing.assert_allclose(one["logits"][0, 0], full["logits"][0, i], rtol=0, atol=1e-10)
        np.testing.assert_allclose(one["node_k"][:, 0, 0], full["node_k"][:, 0, i], rtol=0, atol=1e-10)
        ck, cv, lens = tg.commit(ck, cv, lens, one["node_k"], one["node_v"], [0], np.full((1, 1), -1))
    assert lens[0] == n + m


def test_tree_leaf_equals_substituted_chain():
    """In a two-branch tree the rank-1 leaf of depth d sees only the spine above
    it, so its logits are those of the chain whose depth-d token is the leaf's."""
    cfg, w = _tiny()
    n, depth, beta = 9, 5, 2
    ck, cv = _ctx(cfg, n, 32)
    topk = synth.make_random_topk(cfg.with_(batch=1, block=depth + 1, branch=beta), seed=3)
    tree = oracle.build_tree(topk, [11], [n])
    res = tg.verify_forward(cfg, w, tree["node_token"], tree["node_pos"], tree["ancestor_mask"], [n], ck, cv)
    spine = [11] + [int(topk[0, d, 0]) for d in range(depth)]
    for d in range(1, depth + 1):
        leaf = 1 + (d - 1) * beta + 1
        toks = spine[:d] + [int(topk[0, d - 1, 1])]
        tok, pos, mask = _chain(toks, n)
        ch = tg.verify_forward(cfg, w, tok, pos, mask, [n], ck, cv)
        np.testing.assert_allclose(res["logits"][0, leaf], ch["logits"][0, d], rtol=0, atol=1e-10)
        # and the spine node of depth d is the chain's node d
        full = tg.verify_forward(cfg, w, *_chain(spine, n), [n], ck, cv)
        np.testing.assert_allclose(res["logits"][0, 1 + (d - 1) * beta], full["logits"][0, d], rtol=0, atol=1e-10)


def test_commit_then_bonus_continues_the_accepted_path():
    """Commit a tree path that ends on a leaf, then run the bonus token alone: its
    logits are the chain [path..., bonus]'s last-node logits."""
    cfg, w = _tiny()
    n, depth, beta = 12, 4, 3
    ck, cv = _ctx(cfg, n, 40)
    topk = synth.make_random_topk(cfg.with_(batch=1, block=depth + 1, branch=beta), seed=5)
    tree = oracle.build_tree(topk, [21], [n])
    res = tg.verify_forward(cfg, w, tree["node_token"], tree["node_pos"], tree["ancestor_mask"], [n], ck, cv)
    acc_nodes = np.array([[1, 1 + beta, 1 + 2 * beta + 2, -1]])    # spine, spine, then a leaf
    ck2, cv2, lens = tg.commit(ck, cv, [n], res["node_k"], res["node_v"], [3], acc_nodes)
    assert lens[0] == n + 4
    for d, node in enumerate([0, 1, 1 + beta, 1 + 2 * beta + 2]):
        np.testing.assert_array_equal(ck2[:, 0, n + d], res["node_k"][:, 0, node])
    np.testing.assert_array_equal(ck2[:, 0, :n], ck[:, 0, :n])                   # context untouched
    bonus = 77
    one = tg.verify_forward(cfg, w, [[bonus]], [[n + 4]], np.ones((1, 1, 1), np.uint8), lens, ck2, cv2)
    path = [int(tree["node_token"][0, k]) for k in (0, 1, 1 + beta, 1 + 2 * beta + 2)] + [bonus]
    ch = tg.verify_forward(cfg, w, *_chain(path, n), [n], ck, cv)
    np.testing.assert_allclose(one["logits"][0, 0], ch["logits"][0, 4], rtol=0, atol=1e-10)


def test_zero_attention_and_ffn_outputs_closed_form():
    cfg = synth.get_config("tiny_target").with_(n_layers=3)
    w = synth.make_target_weights(cfg, seed=2, gain_std=0.1, zero_wo_wdown=True)
    n = 10
    ck, cv = _ctx(cfg, n, 16)
    toks = [5, 4095, 17, 5]
    res = tg.verify_forward(cfg, w, *_chain(toks, n), [n], ck, cv)
    e = np.asarray(w["embed"], F64)[toks]
    want = oracle.rms_norm(e, w["final_norm"], cfg.rms_eps) @ np.asarray(w["lm_head"], F64).T
    np.testing.assert_allclose(res["logits"][0], want, rtol=0, atol=1e-12)
