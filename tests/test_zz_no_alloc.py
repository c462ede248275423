"""The acceptance entry point that allocates nothing (domino_verify_accept_noalloc):
through the C ABI, its outputs must equal domino_verify_accept's bit for bit on the
same tree and target logits, on two calls in a row (the second smaller, so stale
partials of the first would show).  Its rejection of sizes beyond the fixed
scratch is checked on the CPU (test_abi.py)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(batch, beta, V, seed, dtype):
    cfg = synth.get_config("qwen3_8b").with_(batch=batch, branch=beta, vocab=V)
    topk = synth.make_random_topk(cfg, seed=seed)
    tree = oracle.build_tree(topk, np.arange(batch, dtype=np.int32), np.full(batch, 9, np.int32))
    lg = synth.make_target_logits(cfg, tree["node_token"], tree["node_parent"], seed=seed, dtype=dtype)
    return cfg, tree, lg


def _run(tree, lg_t, block, noalloc):
    from paper_2605_29707_amd import binding as bd
    dev = lg_t.device
    bs, nn, V = lg_t.shape
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    acc = torch.full((bs,), -7, dtype=torch.int32, device=dev)
    nodes = torch.full((bs, block - 1), -7, dtype=torch.int32, device=dev)
    out = torch.full((bs, block), -7, dtype=torch.int32, device=dev)
    if noalloc:
        err = torch.full((1,), 123, dtype=torch.int32, device=dev)
        bd.domino_verify_accept_noalloc(t(tree["node_token"]), t(tree["node_parent"]), lg_t, block, acc, nodes,
                                        out, err)
        torch.cuda.synchronize()
        e = int(err.item())
    else:
        ws = torch.empty(bd.domino_verify_workspace_bytes(bs, nn, V), dtype=torch.uint8, device=dev)
        bd.domino_verify_accept(t(tree["node_token"]), t(tree["node_parent"]), lg_t, block, acc, nodes, out, ws)
        torch.cuda.synchronize()
        e = bd.domino_workspace_error(ws)
    return {"accept_len": acc.cpu().numpy(), "accepted_nodes": nodes.cpu().numpy(),
            "out_tokens": out.cpu().numpy(), "err": e}


def test_noalloc_accept_matches_workspace_accept_twice():
    # first a large call (bs 8, beta 4: 61 nodes at the full vocabulary), then a smaller one
    cases = [(8, 4, 151936, 0, "bf16"), (2, 1, 50000, 1, "f32")]
    for batch, beta, V, seed, dtype in cases:
        log(f"noalloc acceptance: batch {batch}, beta {beta}, vocab {V}, {dtype}")
        cfg, tree, lg = _case(batch, beta, V, seed, dtype)
        lt = torch.from_numpy(lg).to("cuda:0").to(torch.bfloat16 if dtype == "bf16" else torch.float32)
        want = _run(tree, lt, cfg.block, noalloc=False)
        got = _run(tree, lt, cfg.block, noalloc=True)
        assert want["err"] == 0 and got["err"] == 0
        for k in ("accept_len", "accepted_nodes", "out_tokens"):
            np.testing.assert_array_equal(got[k], want[k], err_msg=k)
        ref = oracle.verify_accept(tree["node_token"], tree["node_parent"], lg, cfg.block)
        for k in ref:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
        log(f"  tau {list(got['accept_len'] + 1)}")

