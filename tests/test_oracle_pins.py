"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these re-type the oracle's own formulas: each compares against an
independent library routine (torch's fp64 GRUCell/GRU and scaled-dot-product
attention), a closed form, an invariant stated by the paper, or brute force on
tiny inputs.  Parity of the backbone layer's internal wiring (which norm sits
where) has no pin beyond its written reading: the paper names the DFlash
architecture without its internals ("parity unpinned" for that wiring; the
closed-form special cases below still pin the residual/norm/LM-head skeleton).
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_cfg(**kw):
    base = dict(hidden=64, n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
                vocab=97, gru_hidden=24, rank=8, dtype="f32", batch=2, ctx=11, branch=2)
    base.update(kw)
    return synth.DominoConfig("pin", **base)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_closed_form_constant_vector():
    # x = c * 1 -> each output = g * c / sqrt(c^2 + eps)
    for c in (-3.0, 0.25, 7.5):
        x = np.full((1, 10), c)
        g = np.arange(1, 11, dtype=float)
        got = O.rms_norm(x, g, 1e-6)
        np.testing.assert_allclose(got[0], g * c / np.sqrt(c * c + 1e-6), rtol=1e-14)


def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 33))
    y = O.rms_norm(x, np.ones(33), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-13)
    np.testing.assert_allclose(O.rms_norm(17.0 * x, np.ones(33), 0.0), y, rtol=1e-12)


# ---------------------------------------------------------------- RoPE
def test_rope_identity_at_position_zero():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 2, 8))
    np.testing.assert_array_equal(O.rope(x, np.zeros(3), 1e6), x)


def test_rope_equals_complex_rotation_of_half_pairs():
    # independent formulation: z_i = x_i + 1j x_{i+d/2} multiplied by exp(1j p w_i)
    rng = np.random.default_rng(2)
    d, theta = 8, 1e6
    x = rng.standard_normal((4, 1, d))
    pos = np.array([0.0, 1.0, 17.0, 1025.0])
    z = x[..., : d // 2] + 1j * x[..., d // 2:]
    w = theta ** (-np.arange(0, d, 2) / d)
    zr = z * np.exp(1j * pos[:, None, None] * w[None, None, :])
    want = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(O.rope(x, pos, theta), want, rtol=1e-12, atol=1e-12)


def test_rope_preserves_norm_and_is_relative():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))
    r = O.rope(q, np.array([5.0]), 1e4)
    np.testing.assert_allclose(np.linalg.norm(r), np.linalg.norm(q), rtol=1e-13)
    s1 = np.sum(O.rope(q, np.array([9.0]), 1e4) * O.rope(k, np.array([4.0]), 1e4))
    s2 = np.sum(O.rope(q, np.array([105.0]), 1e4) * O.rope(k, np.array([100.0]), 1e4))
    assert abs(s1 - s2) < 1e-11


# ---------------------------------------------------------------- attention
@pytest.mark.parametrize("nq,nkv,lk", [(4, 2, 13), (8, 8, 5), (32, 8, 40)])
def test_attention_matches_torch_sdpa(nq, nkv, lk):
    rng = np.random.default_rng(nq + lk)
    dh, lq = 16, 6
    q = rng.standard_normal((lq, nq, dh))
    k = rng.standard_normal((lk, nkv, dh))
    v = rng.standard_normal((lk, nkv, dh))
    got = O.attention(q, k, v)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(nq // nkv, dim=0)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(nq // nkv, dim=0)[None]
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_attention_identical_keys_is_mean_of_values():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((3, 2, 8))
    k = np.repeat(rng.standard_normal((1, 1, 8)), 9, axis=0)
    v = rng.standard_normal((9, 1, 8))
    got = O.attention(q, k, v)
    np.testing.assert_allclose(got, np.broadcast_to(v.mean(axis=0), got.shape), rtol=1e-12)


# ---------------------------------------------------------------- GRU
def test_gru_cell_matches_torch_grucell():
    rng = np.random.default_rng(5)
    d, ds = 12, 7
    w = {"gru_w_ih": rng.standard_normal((3 * ds, d)), "gru_w_hh": rng.standard_normal((3 * ds, ds)),
         "gru_b_ih": rng.standard_normal(3 * ds), "gru_b_hh": rng.standard_normal(3 * ds)}
    cell = torch.nn.GRUCell(d, ds).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(w["gru_w_ih"]))
        cell.weight_hh.copy_(torch.from_numpy(w["gru_w_hh"]))
        cell.bias_ih.copy_(torch.from_numpy(w["gru_b_ih"]))
        cell.bias_hh.copy_(torch.from_numpy(w["gru_b_hh"]))
    h = rng.standard_normal(ds)
    for _ in range(4):
        e = rng.standard_normal(d)
        want = cell(torch.from_numpy(e)[None], torch.from_numpy(h)[None])[0].detach().numpy()
        got = O.gru_cell(w, e, h)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)
        h = got


def test_gru_cell_zero_weights_closed_form():
    rng = np.random.default_rng(6)
    ds, d = 5, 3
    bi, bh = rng.standard_normal(3 * ds), rng.standard_normal(3 * ds)
    w = {"gru_w_ih": np.zeros((3 * ds, d)), "gru_w_hh": np.zeros((3 * ds, ds)), "gru_b_ih": bi, "gru_b_hh": bh}
    h = rng.standard_normal(ds)
    z = 1 / (1 + np.exp(-(bi[ds:2 * ds] + bh[ds:2 * ds])))
    r = 1 / (1 + np.exp(-(bi[:ds] + bh[:ds])))
    want = (1 - z) * np.tanh(bi[2 * ds:] + r * bh[2 * ds:]) + z * h
    np.testing.assert_allclose(O.gru_cell(w, rng.standard_normal(d), h), want, rtol=1e-13)


# ---------------------------------------------------------------- selection order
def _brute_top(vals, beta):
    items = [(-np.inf if np.isnan(v) else v, i) for i, v in enumerate(vals)]
    chosen = []
    for _ in range(beta):
        best = None
        for v, i in items:
            if i in chosen:
                continue
            if best is None or v > best[0] or (v == best[0] and i < best[1]):
                best = (v, i)
        chosen.append(best[1])
    return chosen


def test_top_beta_brute_force_with_ties_and_nan():
    rng = np.random.default_rng(7)
    for trial in range(60):
        n = int(rng.integers(3, 40))
        v = rng.integers(-3, 4, size=n).astype(float)   # many exact ties
        if trial % 3 == 0:
            v[rng.integers(0, n, size=2)] = np.nan
        beta = int(rng.integers(1, min(n, 8) + 1))
        ids, _ = O.top_beta(v, beta)
        assert list(ids) == _brute_top(v, beta)
        assert O.argmax_total(v) == _brute_top(v, 1)[0]


def test_argmax_all_nan_and_neg_inf():
    assert O.argmax_total(np.array([np.nan, np.nan, np.nan])) == 0
    assert O.argmax_total(np.array([-np.inf, np.nan, -np.inf])) == 0
    assert O.argmax_total(np.array([np.nan, -5.0, np.nan])) == 1


# ---------------------------------------------------------------- tree
@pytest.mark.parametrize("beta", [1, 2, 4])
def test_tree_invariants(beta):
    cfg = tiny_cfg(branch=beta, batch=3)
    topk = synth.make_random_topk(cfg, seed=beta)
    anchor = np.array([5, 6, 7], np.int32)
    lens = np.array([0, 11, 4], np.int32)
    t = O.build_tree(topk, anchor, lens)
    nn = 1 + 15 * beta
    assert t["node_token"].shape == (3, nn)
    for b in range(3):
        par, dep, tok = t["node_parent"][b], t["node_depth"][b], t["node_token"][b]
        assert par[0] == -1 and dep[0] == 0 and tok[0] == anchor[b]
        for i in range(1, nn):
            assert dep[i] == dep[par[i]] + 1                   # parent one level up
            assert t["node_pos"][b, i] == lens[b] + dep[i]
            assert par[i] == 0 or (par[i] - 1) % beta == 0     # only spine nodes have children
        for d in range(1, 16):                                  # distinct tokens per depth
            toks = tok[dep == d]
            assert len(toks) == beta and len(set(toks.tolist())) == beta
        # mask is the reflexive-transitive closure of the parent relation
        m = t["ancestor_mask"][b].astype(bool)
        closure = np.eye(nn, dtype=bool)
        for i in range(nn):
            closure[i, par[i]] = par[i] >= 0
        for _ in range(16):
            closure = closure | ((closure.astype(int) @ closure.astype(int)) > 0)
        assert (m == closure).all()
    if beta == 1:
        # chain: node i's parent is i-1
        assert (t["node_parent"][:, 1:] == np.arange(15)).all()


# ---------------------------------------------------------------- acceptance
def _brute_accept(tok, par, logits):
    nn = len(tok)
    R = [O.argmax_total(logits[m]) for m in range(nn)]
    best, best_d = 0, 0
    for i in range(nn):
        path, k = [], i
        while k > 0:
            path.append(k)
            k = par[k]
        if all(tok[c] == R[par[c]] for c in path) and len(path) > best_d:
            best, best_d = i, len(path)
    return best_d, R[best]


@pytest.mark.parametrize("beta", [1, 3])
def test_acceptance_brute_force_tiny_vocab(beta):
    V = 6      # tiny vocabulary: many chance matches
    cfg = tiny_cfg(vocab=V, branch=beta, batch=1)
    for seed in range(40):
        topk = synth.make_random_topk(cfg, seed=seed, vocab=V)
        t = O.build_tree(topk, np.array([1]), np.array([0]))
        for kind in ("zipf", "normal"):
            lg = synth.make_target_logits(cfg, t["node_token"], t["node_parent"], seed=seed,
                                          kind=kind, dtype="f32", vocab=V)
            res = O.verify_accept(t["node_token"], t["node_parent"], lg)
            a, bonus = _brute_accept(t["node_token"][0], t["node_parent"][0], lg[0])
            assert res["accept_len"][0] == a
            assert 1 <= a + 1 <= cfg.block                      # tau in [1, gamma+1]
            assert res["out_tokens"][0, a] == bonus
            assert (res["out_tokens"][0, a + 1:] == -1).all()
            assert (res["accepted_nodes"][0, a:] == -1).all()


def test_acceptance_beta1_is_longest_prefix():
    cfg = tiny_cfg(vocab=50, branch=1, batch=1)
    for seed in range(20):
        topk = synth.make_random_topk(cfg, seed=seed, vocab=50)
        t = O.build_tree(topk, np.array([3]), np.array([0]))
        lg = synth.make_target_logits(cfg, t["node_token"], t["node_parent"], seed=seed,
                                      dtype="f32", vocab=50)
        res = O.verify_accept(t["node_token"], t["node_parent"], lg)
        draft = topk[0, :, 0]
        R = [int(np.argmax(lg[0, m])) for m in range(16)]       # unique maxima (zipf rows)
        a = 0
        while a < 15 and draft[a] == R[a]:
            a += 1
        assert res["accept_len"][0] == a and res["out_tokens"][0, a] == R[a]


# ---------------------------------------------------------------- architecture size
def test_head_param_count_is_56M_at_qwen3_8b_shape():
    gold = json.load(open(os.path.join(GOLDEN, "paper_constants.json")))
    cfg = synth.get_config("qwen3_8b")
    assert (cfg.block, cfg.n_layers, cfg.gru_hidden, cfg.rank) == (
        gold["block"], gold["backbone_layers"], gold["gru_hidden"], gold["rank"])
    n = synth.head_param_count(cfg)
    assert n == 55_934_976
    assert round(n / 1e6) == gold["head_params_millions_rounded"]
    assert round(synth.head_param_count(cfg, with_gru_bias=True) / 1e6) == 56
    # a GRU fed d_s-wide inputs, or a correction without the full vocab-wide W2,
    # would not give 56M
    ds, d, r, V = 1024, 4096, 256, 151936
    assert round((6 * ds * ds + r * (d + ds) + V * r) / 1e6) != 56
    assert round((3 * ds * d + 3 * ds * ds + r * (d + ds) + d * r) / 1e6) != 56


# ---------------------------------------------------------------- Domino head structure
def _tiny_step(cfg, seed=0, **wkw):
    w = O.as_f64_weights(synth.make_weights(cfg, seed=seed, gain_std=0.1, **wkw))
    inp = synth.make_inputs(cfg, seed=seed)
    return w, inp


def test_head_state_matches_torch_gru_over_prefix():
    # S_{j-1} must equal a GRU run over E(anchor), E(y_1), ..., E(y_{j-1})
    cfg = tiny_cfg(batch=1)
    w, inp = _tiny_step(cfg)
    forced = synth.make_forced_tokens(cfg, seed=3)
    h = np.zeros((15, cfg.hidden))
    lb = np.zeros((15, cfg.vocab))
    _, _, _, states, _ = O.domino_head(cfg, w, h, lb, inp["anchor"][0], 1, forced[0])
    gru = torch.nn.GRU(cfg.hidden, cfg.gru_hidden).double()
    with torch.no_grad():
        gru.weight_ih_l0.copy_(torch.from_numpy(w["gru_w_ih"]))
        gru.weight_hh_l0.copy_(torch.from_numpy(w["gru_w_hh"]))
        gru.bias_ih_l0.copy_(torch.from_numpy(w["gru_b_ih"]))
        gru.bias_hh_l0.copy_(torch.from_numpy(w["gru_b_hh"]))
    seq = [int(inp["anchor"][0])] + [int(t) for t in forced[0, :14]]
    e = torch.from_numpy(w["embed"][seq])[:, None, :]
    out, _ = gru(e)
    np.testing.assert_allclose(states, out[:, 0, :].detach().numpy(), rtol=1e-11, atol=1e-12)


def test_perturbation_causality():
    # L_1..L_i depend only on tokens before i: changing forced tokens at and
    # after i leaves them unchanged; changing y_{i-1} changes L_i.
    cfg = tiny_cfg(batch=1)
    w, inp = _tiny_step(cfg)
    forced = synth.make_forced_tokens(cfg, seed=1)
    base = O.draft_step(cfg, w, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], 2, forced)
    for i in (0, 5, 14):
        f2 = forced.copy()
        f2[0, i:] = (f2[0, i:] + 1 + np.arange(15 - i)) % cfg.vocab
        alt = O.draft_step(cfg, w, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], 2, f2)
        np.testing.assert_array_equal(alt["final_logits"][0, : i + 1], base["final_logits"][0, : i + 1])
        np.testing.assert_array_equal(alt["base_logits"], base["base_logits"])
        if i + 1 < 15:
            assert np.abs(alt["final_logits"][0, i + 1] - base["final_logits"][0, i + 1]).max() > 0


def test_anchor_reaches_first_position():
    cfg = tiny_cfg(batch=1)
    w, _ = _tiny_step(cfg)
    h = np.random.default_rng(0).standard_normal((15, cfg.hidden))
    lb = np.zeros((15, cfg.vocab))
    a = O.domino_head(cfg, w, h, lb, 3, 1)[2]
    b = O.domino_head(cfg, w, h, lb, 4, 1)[2]
    assert np.abs(a[0] - b[0]).max() > 0


def test_zero_head_reproduces_backbone():
    cfg = tiny_cfg(batch=2, branch=3)
    w, inp = _tiny_step(cfg, zero_head=True)
    r = O.draft_step(cfg, w, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], 3)
    np.testing.assert_array_equal(r["final_logits"], r["base_logits"])
    for b, j in itertools.product(range(2), range(15)):
        ids, _ = O.top_beta(r["base_logits"][b, j], 3)
        assert (r["topk_ids"][b, j] == ids).all()


def test_correction_split_W1_columns():
    # W1 columns [H | S]: zeroing the S half makes dL independent of S, and the H half of H
    rng = np.random.default_rng(9)
    d, ds, r, V = 6, 5, 4, 7
    w = {"w1": rng.standard_normal((r, d + ds)), "w2": rng.standard_normal((V, r))}
    h, s1, s2 = rng.standard_normal(d), rng.standard_normal(ds), rng.standard_normal(ds)
    wS0 = dict(w, w1=np.concatenate([w["w1"][:, :d], np.zeros((r, ds))], axis=1))
    np.testing.assert_array_equal(O.correction(wS0, h, s1), O.correction(wS0, h, s2))
    wH0 = dict(w, w1=np.concatenate([np.zeros((r, d)), w["w1"][:, d:]], axis=1))
    np.testing.assert_array_equal(O.correction(wH0, h, s1), O.correction(wH0, 2 * h, s1))
    assert np.abs(O.correction(w, h, s1) - O.correction(w, h, s2)).max() > 0


# ---------------------------------------------------------------- backbone closed forms
def test_backbone_with_zero_output_projections_closed_form():
    # W_o = W_down = 0: the residual stream stays the block embedding, so
    # H_j = RMSNorm(E[MASK]) for every draft row and all base-logit rows agree
    cfg = tiny_cfg(batch=1)
    w, inp = _tiny_step(cfg, zero_wo_wdown=True)
    r = O.draft_step(cfg, w, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], 1)
    e = w["embed"][cfg.mask_id]
    hm = e / np.sqrt(np.mean(e * e) + cfg.rms_eps) * w["final_norm"]
    want = w["lm_head"] @ hm
    for j in range(15):
        np.testing.assert_allclose(r["base_logits"][0, j], want, rtol=1e-12, atol=1e-14)


def test_backbone_ignores_context_beyond_ctx_len_and_forced_tokens():
    cfg = tiny_cfg(batch=1)
    w, inp = _tiny_step(cfg)
    lens = np.array([6], np.int32)
    r1 = O.draft_step(cfg, w, inp["anchor"], lens, inp["ctx_k"], inp["ctx_v"], 1)
    k2, v2 = inp["ctx_k"].copy(), inp["ctx_v"].copy()
    k2[:, :, 6:] = 1e3
    v2[:, :, 6:] = -1e3
    f = synth.make_forced_tokens(cfg, seed=5)
    r2 = O.draft_step(cfg, w, inp["anchor"], lens, k2, v2, 1, f)
    np.testing.assert_array_equal(r1["base_logits"], r2["base_logits"])


def test_backbone_empty_context_is_block_self_attention():
    # ctx_len = 0: each layer's attention is plain attention over the block rows only
    cfg = tiny_cfg(batch=1)
    w, inp = _tiny_step(cfg)
    r = O.draft_step(cfg, w, inp["anchor"], np.array([0], np.int32), inp["ctx_k"], inp["ctx_v"], 1)
    k2 = np.full_like(inp["ctx_k"], np.nan)
    r2 = O.draft_step(cfg, w, inp["anchor"], np.array([0], np.int32), k2, k2, 1)
    np.testing.assert_array_equal(r["base_logits"], r2["base_logits"])
    assert np.isfinite(r["base_logits"]).all()


def test_context_projection_matches_layer_kv():
    # a context row projected from hidden state c at position p carries exactly the
    # K the layer's own projection gives a row whose normed input is c
    cfg = tiny_cfg(batch=1)
    w, _ = _tiny_step(cfg)
    lw = w["layers"][0]
    rng = np.random.default_rng(11)
    c = rng.standard_normal((3, cfg.hidden))
    k, v = O.project_context_kv(cfg, lw, c, np.array([0.0, 1.0, 2.0]))
    kk = (c @ lw["wk"].T).reshape(3, cfg.n_kv_heads, cfg.head_dim)
    np.testing.assert_allclose(k[0], O.rms_norm(kk[0], lw["k_norm"], cfg.rms_eps), rtol=1e-13)
    np.testing.assert_allclose(np.linalg.norm(k, axis=-1),
                               np.linalg.norm(O.rms_norm(kk, lw["k_norm"], cfg.rms_eps), axis=-1),
                               rtol=1e-12)
    np.testing.assert_allclose(v, (c @ lw["wv"].T).reshape(3, cfg.n_kv_heads, cfg.head_dim), rtol=1e-13)


# ---------------------------------------------------------------- context fusion
def _drafter_own_params(cfg):
    """Parameters the drafter trains itself: backbone layers, final norm and the
    context-fusion map (the embedding and LM head are the target's, frozen)."""
    s = synth.weight_shapes(cfg)
    n = sum(int(np.prod(v)) for lw in s["layers"] for v in lw.values())
    n += int(np.prod(s["final_norm"]))
    if "ctx_fc" in s:
        n += int(np.prod(s["ctx_fc"]))
    return n


def test_context_fusion_makes_the_head_5_3_percent_of_the_drafter():
    # Sec. 1: the head adds 56M parameters, +5.3% over the drafter without it.
    # Five fused target layers (an ~84M map) give 5.33%, the fusion width
    # closest to 5.3%; without a fusion map the head would be 5.8%.
    gold = json.load(open(os.path.join(GOLDEN, "paper_constants.json")))
    pct = gold["head_params_relative_percent"]
    cfg = synth.get_config("qwen3_8b")
    assert cfg.ctx_fuse_layers == 5
    head = synth.head_param_count(cfg)
    assert round(int(np.prod(synth.weight_shapes(cfg)["ctx_fc"])) / 1e6) == 84
    share = {k: 100 * head / _drafter_own_params(cfg.with_(ctx_fuse_layers=k)) for k in range(9)}
    assert round(share[5], 1) == pct
    assert min(share, key=lambda k: abs(share[k] - pct)) == 5
    assert round(share[0], 1) == 5.8


def _fused_vs_plain(k, fc_blocks, hidden_blocks):
    """Draft step with k fused layers and ctx_fc = [fc_blocks...] against the
    plain (unfused) step fed the given hidden states."""
    cfg = tiny_cfg(batch=1, ctx=9, ctx_from_hidden=True, ctx_fuse_layers=k)
    plain = cfg.with_(ctx_fuse_layers=0)
    w, inp = _tiny_step(plain)
    d = cfg.hidden
    rng = np.random.default_rng(21)
    blocks = [rng.standard_normal((1, 9, d)) for _ in range(k)]
    cat = np.concatenate(blocks, axis=-1)
    wf = dict(w)
    wf["ctx_fc"] = np.concatenate([np.asarray(b, np.float64) for b in fc_blocks], axis=1)
    lens = np.array([9], np.int32)
    r = O.draft_step(cfg, wf, inp["anchor"], lens, inp["ctx_k"], inp["ctx_v"], 1, ctx_hidden=cat)
    r2 = O.draft_step(plain, w, inp["anchor"], lens, inp["ctx_k"], inp["ctx_v"], 1,
                      ctx_hidden=hidden_blocks(blocks))
    return r, r2


@pytest.mark.parametrize("pick", [0, 1, 2])
def test_context_fusion_selecting_one_layer_is_that_layer(pick):
    # ctx_fc = [0 .. I .. 0] picks layer `pick` of the concatenation: the step
    # equals the unfused step fed that layer's hidden states
    d = tiny_cfg().hidden
    fc = [np.eye(d) if i == pick else np.zeros((d, d)) for i in range(3)]
    r, r2 = _fused_vs_plain(3, fc, lambda b: b[pick])
    np.testing.assert_allclose(r["base_logits"], r2["base_logits"], rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(r["topk_ids"], r2["topk_ids"])


def test_context_fusion_equal_weights_is_the_mean_of_layers():
    d = tiny_cfg().hidden
    r, r2 = _fused_vs_plain(3, [np.eye(d) / 3] * 3, lambda b: (b[0] + b[1] + b[2]) / 3)
    np.testing.assert_allclose(r["base_logits"], r2["base_logits"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(r["final_logits"], r2["final_logits"], rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------- SiLU, the correction and SwiGLU
# Logistic values written out to 16 digits: sigma(1) = 1 / (1 + e^-1),
# sigma(2) = 1 / (1 + e^-2), sigma(-1) = 1 - sigma(1).
SIGMA_1 = 0.7310585786300049
SIGMA_2 = 0.8807970779778823
SIGMA_M1 = 0.2689414213699951


def test_silu_matches_torch_and_closed_forms():
    # SiLU(x) = x * sigma(x) (the correction equation of Sec. 4.1.2 and the FFN's gate)
    x = np.linspace(-30.0, 30.0, 241)
    want = torch.nn.functional.silu(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(O.silu(x), want, rtol=1e-14, atol=1e-300)
    assert O.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(O.silu(np.array([1.0, 2.0, -1.0])), [SIGMA_1, 2 * SIGMA_2, -SIGMA_M1], rtol=1e-15)
    # SiLU(x) -> x for large x, -> 0 from below for very negative x
    np.testing.assert_allclose(O.silu(np.array([40.0]))[0], 40.0, rtol=1e-15)
    v = O.silu(np.array([-40.0]))[0]
    assert v < 0 and abs(v) < 1e-15


def test_correction_closed_form_with_selector_rows():
    # W1 rows pick single entries of [H; S], W2 mixes the two rank rows, so
    # dL = W2 SiLU(W1 [H; S]) is known by hand: pre-activations (1, -1) give
    # u = (sigma(1), -sigma(-1)).  Sigmoid in place of SiLU, or no activation,
    # gives other values.
    d, ds = 2, 2
    w1 = np.zeros((2, d + ds))
    w1[0, 0] = 1.0          # u_0 from H_0
    w1[1, d + 1] = 2.0      # u_1 from 2 * S_1
    w2 = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    h = np.array([1.0, 5.0])
    s = np.array([7.0, -0.5])
    got = O.correction({"w1": w1, "w2": w2}, h, s)
    np.testing.assert_allclose(got, [SIGMA_1, -SIGMA_M1, SIGMA_1 - SIGMA_M1], rtol=1e-15)


def test_swiglu_ffn_closed_form():
    # One layer with W_o = 0 (attention adds nothing) and a hand-built FFN:
    # x = (1, -1, 1, -1) has unit RMS, so with eps 0 and unit gains the FFN
    # input is x itself.  Unit 0: gate 2*y_0 = 2, up y_1 = -1 -> SiLU(2) * -1;
    # unit 1: gate y_1 = -1, up 3*y_2 = 3 -> SiLU(-1) * 3.  W_down sends unit 0
    # to column 0 and unit 1 to column 3.  Swapping gate and up, or sigmoid in
    # place of SiLU, changes both columns.
    from types import SimpleNamespace
    cfg = SimpleNamespace(n_q_heads=1, n_kv_heads=1, head_dim=4, rms_eps=0.0, rope_theta=1e6)
    rng = np.random.default_rng(21)
    d, ffn = 4, 2
    wg = np.zeros((ffn, d)); wg[0, 0] = 2.0; wg[1, 1] = 1.0
    wu = np.zeros((ffn, d)); wu[0, 1] = 1.0; wu[1, 2] = 3.0
    wd = np.zeros((d, ffn)); wd[0, 0] = 1.0; wd[3, 1] = 1.0
    lw = {"attn_norm": np.ones(d), "wq": rng.standard_normal((4, d)), "wk": rng.standard_normal((4, d)),
          "wv": rng.standard_normal((4, d)), "q_norm": np.ones(4), "k_norm": np.ones(4), "wo": np.zeros((d, 4)),
          "ffn_norm": np.ones(d), "w_gate": wg, "w_up": wu, "w_down": wd}
    x = np.array([[1.0, -1.0, 1.0, -1.0]])
    empty = np.zeros((0, 1, 4))
    got = O.backbone_layer(cfg, lw, x, np.array([0.0]), empty, empty)
    want = [1.0 - 2 * SIGMA_2, -1.0, 1.0, -1.0 - 3 * SIGMA_M1]
    np.testing.assert_allclose(got[0], want, rtol=1e-15, atol=1e-15)
