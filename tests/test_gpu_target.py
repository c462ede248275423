"""GPU parity of the target tree-verify forward and the cache commit through
the C-ABI, against the target oracle.

The trees are built on the GPU by domino_build_tree (the oracle builds its own
from the same top-beta ids; the two are bit-exact, tested elsewhere).
Tolerances: logits and stored K/V at the drafting bar (1e-4 absolute fp32;
2e-2 bf16, K/V stored in bf16 also within bf16 rounding), cache moves and
context lengths bit-exact.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import log

tg = oracle.target_oracle
pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_29707_amd import binding as bd  # noqa: E402

DEV = torch.device("cuda:0")


def _t(a, dt=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    return t if dt is None else t.to(dt)


class Target:
    def __init__(self, cfg, w):
        self.cfg = cfg
        self.dw = bd.to_device_weights(w, cfg, DEV)
        self.model = bd.DominoModel(cfg, self.dw, target=True)
        self.kvdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def tree(self, topk, anchor, lens):
        bs, depth, beta = topk.shape
        nn = 1 + depth * beta
        outs = [torch.empty(bs, nn, dtype=torch.int32, device=DEV) for _ in range(4)]
        mask = torch.empty(bs, nn, nn, dtype=torch.uint8, device=DEV)
        bd.domino_build_tree(_t(topk), _t(anchor, torch.int32), _t(lens, torch.int32), *outs, ancestor_mask=mask)
        return outs[0], outs[1], outs[3], mask

    def verify(self, tok, pos, mask, lens, ck, cv, max_ctx, out_dtype=torch.float32):
        bs, nn = tok.shape
        ws = torch.empty(bd.domino_target_workspace_bytes(self.model, bs, nn, max_ctx), dtype=torch.uint8,
                         device=DEV)
        lg = torch.empty(bs, nn, self.cfg.vocab, dtype=out_dtype, device=DEV)
        bd.domino_target_verify(self.model, tok, pos, mask, _t(lens, torch.int32), ck, cv, max_ctx, lg, ws)
        torch.cuda.synchronize()
        return lg, ws


def _inputs(cfg, lens, max_ctx, seed):
    inp = synth.make_inputs(cfg.with_(batch=len(lens)), seed=seed, ctx_lens=np.array(lens, np.int32), max_ctx=max_ctx)
    return inp


@pytest.mark.parametrize("dtype,beta,lens", [("f32", 1, [100]), ("f32", 2, [128 - 40, 3, 0]),
                                             ("f32", 4, [60, 17]), ("bf16", 2, [50, 90])])
def test_tiny_verify_against_oracle(dtype, beta, lens):
    cfg = synth.get_config("tiny_target").with_(dtype=dtype)
    w = synth.make_target_weights(cfg, seed=31, gain_std=0.1)
    depth = 15
    nn = 1 + depth * beta
    max_ctx = max(lens) + nn + 5
    inp = _inputs(cfg, lens, max_ctx, seed=31)
    bs = len(lens)
    topk = synth.make_random_topk(cfg.with_(batch=bs, block=depth + 1, branch=beta), seed=31)
    run = Target(cfg, w)
    tok, par, pos, mask = run.tree(topk, inp["anchor"], inp["ctx_lens"])
    ck, cv = _t(inp["ctx_k"], run.kvdt), _t(inp["ctx_v"], run.kvdt)
    lg, ws = run.verify(tok, pos, mask, inp["ctx_lens"], ck, cv, max_ctx)
    assert bd.domino_workspace_error(ws) == 0
    tree = oracle.build_tree(topk, inp["anchor"], inp["ctx_lens"])
    np.testing.assert_array_equal(tok.cpu().numpy(), tree["node_token"])
    ref = tg.verify_forward(cfg, w, tree["node_token"], tree["node_pos"], tree["ancestor_mask"], inp["ctx_lens"],
                            inp["ctx_k"], inp["ctx_v"])
    tol = 1e-4 if dtype == "f32" else 2e-2
    err = float(np.abs(lg.cpu().numpy() - ref["logits"]).max())
    got_k, got_v = ck.float().cpu().numpy(), cv.float().cpu().numpy()
    kerr = 0.0
    for b, n in enumerate(lens):
        gk, gv = got_k[:, b, n:n + nn], got_v[:, b, n:n + nn]
        rk, rv = ref["node_k"][:, b], ref["node_v"][:, b]
        slack = np.abs(rk) * 2.0 ** -8 if dtype == "bf16" else 0.0
        assert np.all(np.abs(gk - rk) <= slack + 1e-4) and np.all(np.abs(gv - rv) <= np.abs(rv) * (2.0 ** -8 if dtype == "bf16" else 0) + 1e-4)
        kerr = max(kerr, float(np.abs(gk - rk).max()))
        np.testing.assert_array_equal(got_k[:, b, :n], inp["ctx_k"][:, b, :n])   # context untouched
    log(f"{dtype} beta={beta} lens={lens}: {nn} nodes, max |logits - oracle| = {err:.2e}, node K {kerr:.2e}")
    assert err < tol
    run.model.close()


def test_tiny_cycle_verify_accept_commit_twice():
    """Two full target-side cycles: verify, greedy acceptance on the verify's own
    logits, commit; the second cycle's tree hangs off the first one's bonus
    token.  The oracle runs the same cycles on the GPU's acceptance outcome."""
    cfg = synth.get_config("tiny_target").with_(batch=2)
    w = synth.make_target_weights(cfg, seed=41, gain_std=0.1)
    beta, depth = 2, 15
    nn = 1 + depth * beta
    lens = np.array([40, 70], np.int32)
    max_ctx = 70 + 2 * (nn + 1) + 4
    inp = _inputs(cfg, lens, max_ctx, seed=41)
    run = Target(cfg, w)
    ck, cv = _t(inp["ctx_k"], run.kvdt), _t(inp["ctx_v"], run.kvdt)
    rk, rv = inp["ctx_k"].astype(np.float64), inp["ctx_v"].astype(np.float64)
    anchor, cur = inp["anchor"].copy(), lens.copy()
    for cyc in range(2):
        topk = synth.make_random_topk(cfg.with_(block=depth + 1, branch=beta), seed=50 + cyc)
        # plant the target's own choices on part of the tree so acceptance goes deep: not needed for
        # parity, the walk is exact either way
        tok, par, pos, mask = run.tree(topk, anchor, cur)
        lg, ws = run.verify(tok, pos, mask, cur, ck, cv, max_ctx)
        acc = torch.empty(2, dtype=torch.int32, device=DEV)
        nodes = torch.empty(2, depth, dtype=torch.int32, device=DEV)
        outt = torch.empty(2, depth + 1, dtype=torch.int32, device=DEV)
        vws = torch.empty(bd.domino_verify_workspace_bytes(2, nn, cfg.vocab), dtype=torch.uint8, device=DEV)
        bd.domino_verify_accept(tok, par, lg, depth + 1, acc, nodes, outt, vws)
        new_lens = torch.empty(2, dtype=torch.int32, device=DEV)
        bd.domino_target_commit(run.model, nn, _t(cur, torch.int32), acc, nodes, ck, cv, max_ctx, new_lens, ws)
        torch.cuda.synchronize()
        assert bd.domino_workspace_error(ws) == 0
        tree = oracle.build_tree(topk, anchor, cur)
        ref = tg.verify_forward(cfg, w, tree["node_token"], tree["node_pos"], tree["ancestor_mask"], cur, rk, rv)
        err = float(np.abs(lg.cpu().numpy() - ref["logits"]).max())
        a = oracle.verify_accept(tree["node_token"], tree["node_parent"], lg.cpu().numpy(), depth + 1)
        np.testing.assert_array_equal(acc.cpu().numpy(), a["accept_len"])
        rk, rv, rl = tg.commit(rk, rv, cur, ref["node_k"], ref["node_v"], a["accept_len"], a["accepted_nodes"])
        np.testing.assert_array_equal(new_lens.cpu().numpy(), rl)
        cerr = max(float(np.abs(ck.cpu().numpy()[:, b, :rl[b]] - rk[:, b, :rl[b]]).max()) for b in range(2))
        log(f"cycle {cyc}: accept {a['accept_len'].tolist()} logits err {err:.2e}, committed cache err {cerr:.2e}")
        assert err < 1e-4 and cerr < 1e-4
        anchor = a["out_tokens"][np.arange(2), a["accept_len"]].astype(np.int32)
        cur = rl


def test_commit_moves_rows_and_rejects_bad_paths():
    cfg = synth.get_config("tiny_target").with_(dtype="bf16", n_layers=2, batch=3)
    w = synth.make_target_weights(cfg, seed=44)
    run = Target(cfg, w)
    max_ctx, nn, depth = 64, 9, 4  # depth 4, beta 2
    rng = np.random.default_rng(0)
    ck0 = synth.bf16_round(rng.normal(size=(2, 3, max_ctx, 2, 64)).astype(np.float32))
    cv0 = synth.bf16_round(rng.normal(size=(2, 3, max_ctx, 2, 64)).astype(np.float32))
    ck, cv = _t(ck0, torch.bfloat16), _t(cv0, torch.bfloat16)
    lens = np.array([10, 20, 30], np.int32)
    acc = np.array([4, 2, 3], np.int32)
    nodes = np.array([[1, 3, 5, 8], [2, -1, -1, -1], [1, 3, 2, -1]], np.int32)   # row 2: id 2 at depth 3 is invalid
    nodes[1, 0] = 2
    nodes[1, 1] = 3
    new = torch.empty(3, dtype=torch.int32, device=DEV)
    ws = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    bd.domino_target_commit(run.model, nn, _t(lens), _t(acc), _t(nodes), ck, cv, max_ctx, new, ws)
    torch.cuda.synchronize()
    got_k = ck.float().cpu().numpy()
    assert bd.domino_workspace_error(ws) & bd.DEV_BAD_TREE
    assert new.cpu().numpy().tolist() == [15, 23, 30]
    for b in (0, 1):
        n = lens[b]
        path = [0] + nodes[b, :acc[b]].tolist()
        for d, x in enumerate(path):
            np.testing.assert_array_equal(got_k[:, b, n + d], ck0[:, b, n + x])
        np.testing.assert_array_equal(got_k[:, b, :n], ck0[:, b, :n])
        np.testing.assert_array_equal(got_k[:, b, n + len(path):], ck0[:, b, n + len(path):])
    np.testing.assert_array_equal(got_k[:, 2], ck0[:, 2])   # rejected row untouched
    run.model.close()


def test_qwen3_8b_target_chain_full_size():
    """The 36-layer Qwen3-8B-shaped target over a 16-node chain at context 1024
    (the benchmark's configuration), against the fp64 oracle streamed layer by
    layer on the host."""
    cfg = synth.get_config("qwen3_8b_target")
    log("generating the 36-layer target")
    w = synth.make_target_weights(cfg, seed=0)
    inp = synth.make_inputs(cfg, seed=0, max_ctx=cfg.ctx + 16)
    topk = synth.make_random_topk(cfg.with_(branch=1), seed=0)
    run = Target(cfg, w)
    tok, par, pos, mask = run.tree(topk, inp["anchor"], inp["ctx_lens"])
    ck, cv = _t(inp["ctx_k"], run.kvdt), _t(inp["ctx_v"], run.kvdt)
    lg, ws = run.verify(tok, pos, mask, inp["ctx_lens"], ck, cv, inp["max_ctx"], out_dtype=torch.bfloat16)
    lg2, _ = run.verify(tok, pos, mask, inp["ctx_lens"], ck, cv, inp["max_ctx"], out_dtype=torch.float32)
    assert bd.domino_workspace_error(ws) == 0
    got = lg2.cpu().numpy()
    np.testing.assert_array_equal(lg.float().cpu().numpy(), synth.bf16_round(got.copy()))
    run.model.close()
    del run, ck, cv
    torch.cuda.empty_cache()
    log("oracle (fp64, 36 layers)")
    tree = oracle.build_tree(topk, inp["anchor"], inp["ctx_lens"])
    ref = tg.verify_forward(cfg, w, tree["node_token"], tree["node_pos"], tree["ancestor_mask"], inp["ctx_lens"],
                            inp["ctx_k"], inp["ctx_v"])
    err = float(np.abs(got - ref["logits"]).max())
    log(f"max |logits - oracle| = {err:.2e}")
    assert err < 2e-2
