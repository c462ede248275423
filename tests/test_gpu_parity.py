"""GPU parity of the HIP drafting path (through the C-ABI) against the CPU oracle.

Tolerances: 1e-4 absolute for the fp32 tiny drafter, 2e-2 absolute for bf16
drafters (the stated bar); top-1 and top-beta order must match the oracle
wherever the oracle's adjacent gaps are at least 1e-3.  The oracle is run
teacher-forced on the GPU's own drafted tokens so both sides roll out the same
prefixes.  Trees and acceptance are compared bit-exactly on identical inputs.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import GpuRun, check_against_oracle, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def oracle_for(cfg, w64, inp, gpu, beta, lens=None, forced=None):
    """The oracle teacher-forced on the tokens the GPU step fed back: its own
    top-1 tokens, or `forced` when the GPU step was forced."""
    drafted = gpu["topk_ids"][:, :, 0] if forced is None else forced
    return oracle.draft_step(cfg, w64, inp["anchor"], inp["ctx_lens"] if lens is None else lens,
                             inp["ctx_k"], inp["ctx_v"], beta, forced=drafted,
                             ctx_hidden=inp.get("ctx_hidden"))


def test_tiny_parity_context_from_hidden_states():
    cfg = synth.get_config("tiny")
    log(f"tiny: {cfg}")
    w = synth.make_weights(cfg, seed=1)
    inp = synth.make_inputs(cfg, seed=1)
    n_new = inp["ctx_hidden"].shape[1]
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1, n_new=n_new)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    np.testing.assert_allclose(gpu["ctx_k"], ref["ctx_k"], atol=1e-5, rtol=0)
    n = check_against_oracle(cfg, gpu, ref, 1e-4, 1)
    assert n >= 10
    run.close()


@pytest.mark.parametrize("dtype,k,lens", [("f32", 3, [128]), ("f32", 2, [128, 77]), ("bf16", 5, [101, 128, 64])])
def test_context_fusion_parity(dtype, k, lens):
    """Appended rows of k concatenated target layers ([n_new][k*d]) are fused by
    ctx_fc (a K-split GEMM over k*d columns and the sum of its partials) before
    each layer's K/V projections; ragged context lengths put them at different
    cache positions per batch row."""
    cfg = synth.get_config("tiny").with_(dtype=dtype, ctx_fuse_layers=k, batch=len(lens))
    log(f"context fusion: {dtype} k={k} lens={lens}")
    w = synth.make_weights(cfg, seed=4)
    inp = synth.make_inputs(cfg, seed=4, ctx_lens=np.array(lens, np.int32))
    n_new = inp["ctx_hidden"].shape[1]
    assert inp["ctx_hidden"].shape == (len(lens), n_new, k * cfg.hidden) and n_new == min(lens)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1, n_new=n_new)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    if dtype == "f32":
        np.testing.assert_allclose(gpu["ctx_k"], ref["ctx_k"], atol=1e-5, rtol=0)
        np.testing.assert_allclose(gpu["ctx_v"], ref["ctx_v"], atol=1e-5, rtol=0)
    else:
        # stored in bf16: round-to-nearest error at most 2^-9 relative, plus the fp32 arithmetic
        for got, want in ((gpu["ctx_k"], ref["ctx_k"]), (gpu["ctx_v"], ref["ctx_v"])):
            assert np.all(np.abs(got - want) <= np.abs(want) * 2.0 ** -8 + 1e-4)
    n = check_against_oracle(cfg, gpu, ref, 1e-4 if dtype == "f32" else 2e-2, 1)
    assert n >= 10 * len(lens)
    run.close()


@pytest.mark.parametrize("beta,lens", [(3, [128, 37, 0]), (8, [5, 128, 64]),
                                       (2, [128 - 3 * i for i in range(20)]),
                                       (1, [(37 * i) % 129 for i in range(40)])])
def test_tiny_ragged_batch_branches(beta, lens):
    cfg = synth.get_config("tiny").with_(batch=len(lens), branch=beta, ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=2, gain_std=0.1)
    lens = np.array(lens, np.int32)
    inp = synth.make_inputs(cfg, seed=2, ctx_lens=lens, max_ctx=128)
    log(f"ragged beta={beta} lens={lens.tolist()}")
    run = GpuRun(cfg, w, 128, beta=beta)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, beta)
    check_against_oracle(cfg, gpu, ref, 1e-4, beta)
    run.close()


@pytest.mark.parametrize("batch,beta", [(1, 1), (5, 4), (8, 8), (12, 2)])
def test_tiny_bf16_batches(batch, beta):
    """bf16 storage on the small shape, on both sides of the small-batch rollout
    path (up to 8 rows: one fused state kernel per position; above: the
    three-kernel rollout), with the per-workgroup selection split over waves."""
    cfg = synth.get_config("tiny").with_(dtype="bf16", batch=batch, branch=beta, ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=11, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=11)
    log(f"tiny bf16 batch={batch} beta={beta}")
    run = GpuRun(cfg, w, inp["max_ctx"], beta=beta)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, beta)
    check_against_oracle(cfg, gpu, ref, 2e-2, beta)
    run.close()


@pytest.mark.parametrize("dtype,nq", [("bf16", 4), ("f32", 8), ("bf16", 16)])
def test_long_context_folded_chunks(dtype, nq):
    """16 batch rows over contexts of up to 4096 keys: enough (batch row, kv
    head) pairs that each attention workgroup folds two key chunks into one
    partial with a running softmax (the long-context path); ragged lengths
    leave some workgroups one chunk, some partial chunks and one row with no
    context at all.  nq = 4, 8, 16 over 2 kv heads: 32, 64 and 128 query rows
    per workgroup."""
    lens = [4096, 100, 0, 37, 4095, 64, 65, 2048, 1, 3000, 4000, 129, 127, 500, 4096, 33]
    cfg = synth.get_config("tiny").with_(dtype=dtype, n_q_heads=nq, batch=len(lens), ctx=4096,
                                         ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=13, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=13, ctx_lens=np.array(lens, np.int32), max_ctx=4096)
    log(f"long context: {dtype} nq={nq} bs={len(lens)}")
    run = GpuRun(cfg, w, 4096, beta=1)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    n = check_against_oracle(cfg, gpu, ref, 1e-4 if dtype == "f32" else 2e-2, 1)
    assert n >= 10 * len(lens)
    run.close()


@pytest.mark.parametrize("nq", [8, 16])
def test_bf16_batched_context_one_pass(nq):
    """bf16 cache, head dim 128 and 16 batch rows over 2 kv heads (32 pairs):
    the one-pass context attention (64-key blocks; a run of 128 keys per
    workgroup at nq = 8, and of 192 at nq = 16, whose 8-wave workgroups keep two
    blocks in flight).  The ragged lengths give an empty context, partial
    blocks, block keys split between two workgroups (n = 120, 1016), and
    contexts ending on a workgroup boundary (n = 128, 1024); nq = 8 and 16
    over 2 kv heads: 64 and 128 query rows per workgroup."""
    lens = [1024, 0, 1, 63, 64, 65, 120, 127, 128, 129, 500, 777, 1000, 1008, 1016, 255]
    cfg = synth.get_config("tiny").with_(dtype="bf16", n_q_heads=nq, head_dim=128, batch=len(lens), ctx=1024,
                                         ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=17, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=17, ctx_lens=np.array(lens, np.int32), max_ctx=1024)
    log(f"one-pass context attention: nq={nq} bs={len(lens)}")
    run = GpuRun(cfg, w, 1024, beta=1)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    n = check_against_oracle(cfg, gpu, ref, 2e-2, 1)
    assert n >= 10 * len(lens)
    run.close()


def test_bf16_batched_context_one_pass_long_runs():
    """The one-pass attention over long runs: 64 query rows per workgroup
    (nq = 8 over 2 kv heads), 16 batch rows at a 4096-key context, 320 keys
    (5 blocks) per workgroup.  Ragged lengths: empty, one key, partial blocks,
    contexts ending on a block or a run boundary (64, 320) and one key either
    side of them, block keys split between two runs (n = 310, 3832)."""
    lens = [4096, 0, 1, 63, 64, 65, 319, 320, 321, 310, 2047, 2048, 3000, 4000, 3832, 255]
    cfg = synth.get_config("tiny").with_(dtype="bf16", n_q_heads=8, head_dim=128, batch=len(lens), ctx=4096,
                                         ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=18, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=18, ctx_lens=np.array(lens, np.int32), max_ctx=4096)
    log(f"one-pass context attention, long runs: bs={len(lens)} ctx 4096")
    run = GpuRun(cfg, w, 4096, beta=1)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    n = check_against_oracle(cfg, gpu, ref, 2e-2, 1)
    assert n >= 10 * len(lens)
    run.close()


@pytest.mark.parametrize("nq,block", [(8, 32), (4, 64)])
def test_tiny_large_blocks(nq, block):
    """(n_q / n_kv) * block = 128 query rows per workgroup: the attention uses
    32-key chunks there, and the chunk merge must use the same length (it once
    took 64 whenever n_q / n_kv <= 4)."""
    cfg = synth.get_config("tiny").with_(n_q_heads=nq, block=block, ctx_from_hidden=False, batch=2)
    w = synth.make_weights(cfg, seed=12, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=12, ctx_lens=np.array([128, 45], np.int32), max_ctx=128)
    log(f"tiny nq={nq} block={block}")
    run = GpuRun(cfg, w, 128, beta=1)
    gpu = run.step(inp)
    assert gpu["err"] == 0
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, gpu, 1)
    check_against_oracle(cfg, gpu, ref, 1e-4, 1)
    run.close()


def test_teacher_forcing_and_perturbation_causality():
    cfg = synth.get_config("tiny").with_(ctx_from_hidden=False, batch=2)
    w = synth.make_weights(cfg, seed=3)
    inp = synth.make_inputs(cfg, seed=3)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=2)
    f = synth.make_forced_tokens(cfg, seed=3)
    a = run.step(inp, forced=f)
    ref = oracle.draft_step(cfg, oracle.as_f64_weights(w), inp["anchor"], inp["ctx_lens"], inp["ctx_k"],
                            inp["ctx_v"], 2, forced=f)
    check_against_oracle(cfg, a, ref, 1e-4, 2)
    for i in (0, 6, 14):
        f2 = f.copy()
        f2[:, i:] = (f2[:, i:] + 7) % cfg.vocab
        b = run.step(inp, forced=f2)
        np.testing.assert_array_equal(b["final_logits"][:, : i + 1], a["final_logits"][:, : i + 1])
        np.testing.assert_array_equal(b["states"][:, : i + 1], a["states"][:, : i + 1])
        np.testing.assert_array_equal(b["base_logits"], a["base_logits"])
        if i < 14:
            assert np.abs(b["final_logits"][:, i + 1] - a["final_logits"][:, i + 1]).max() > 0
    run.close()


def test_zero_head_reproduces_backbone_bitwise():
    cfg = synth.get_config("tiny").with_(ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=4, zero_head=True)
    inp = synth.make_inputs(cfg, seed=4)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=4)
    g = run.step(inp)
    np.testing.assert_array_equal(g["final_logits"], g["base_logits"])
    for j in range(cfg.depth):
        ids, _ = oracle.top_beta(g["base_logits"][0, j], 4)
        assert (g["topk_ids"][0, j] == ids).all()
    run.close()


def test_bitwise_repeatable():
    cfg = synth.get_config("tiny").with_(ctx_from_hidden=False, batch=2)
    w = synth.make_weights(cfg, seed=5)
    inp = synth.make_inputs(cfg, seed=5)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=4)
    first = run.step(inp)
    for _ in range(9):
        again = run.step(inp)
        for k in ("topk_ids", "topk_vals", "final_logits", "base_logits", "hidden", "states"):
            np.testing.assert_array_equal(again[k], first[k])
    run.close()


def test_out_of_range_anchor_sets_error_word():
    cfg = synth.get_config("tiny").with_(ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=6)
    inp = synth.make_inputs(cfg, seed=6)
    inp["anchor"] = np.array([cfg.vocab + 5], np.int32)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    g = run.step(inp)
    assert g["err"] & 1
    assert np.isfinite(g["final_logits"]).all()
    inp["anchor"] = np.array([3], np.int32)
    assert run.step(inp)["err"] == 0
    run.close()


# ---------------------------------------------------------------- tree and acceptance
def _tree_gpu(topk, anchor, lens):
    from paper_2605_29707_amd import binding as bd
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bs, depth, beta = topk.shape
    nn = 1 + depth * beta
    outs = [torch.empty(bs, nn, dtype=torch.int32, device=dev) for _ in range(4)]
    mask = torch.empty(bs, nn, nn, dtype=torch.uint8, device=dev)
    bd.domino_build_tree(t(topk), t(anchor), t(lens), *outs, ancestor_mask=mask)
    torch.cuda.synchronize()
    keys = ("node_token", "node_parent", "node_depth", "node_pos")
    res = {k: o.cpu().numpy() for k, o in zip(keys, outs)}
    res["ancestor_mask"] = mask.cpu().numpy()
    return res


@pytest.mark.parametrize("beta", [1, 2, 4, 8])
def test_build_tree_bit_exact(beta):
    cfg = synth.get_config("qwen3_8b").with_(batch=3, branch=beta)
    topk = synth.make_random_topk(cfg, seed=beta)
    anchor = np.array([11, 151000, 0], np.int32)
    lens = np.array([1024, 0, 77], np.int32)
    got = _tree_gpu(topk, anchor, lens)
    want = oracle.build_tree(topk, anchor, lens)
    for k in want:
        np.testing.assert_array_equal(got[k], want[k], err_msg=k)


def _accept_gpu(tok, par, logits_t, block):
    from paper_2605_29707_amd import binding as bd
    dev = logits_t.device
    bs, nn, V = logits_t.shape
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    acc = torch.empty(bs, dtype=torch.int32, device=dev)
    nodes = torch.empty(bs, block - 1, dtype=torch.int32, device=dev)
    out = torch.empty(bs, block, dtype=torch.int32, device=dev)
    ws = torch.empty(bd.domino_verify_workspace_bytes(bs, nn, V), dtype=torch.uint8, device=dev)
    bd.domino_verify_accept(t(tok), t(par), logits_t, block, acc, nodes, out, ws)
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(ws) == 0
    return {"accept_len": acc.cpu().numpy(), "accepted_nodes": nodes.cpu().numpy(),
            "out_tokens": out.cpu().numpy()}


@pytest.mark.parametrize("beta,dtype,kind", [(1, "bf16", "zipf"), (4, "bf16", "zipf"), (4, "f32", "zipf"),
                                             (2, "f32", "normal"), (1, "f32", "normal")])
def test_verify_accept_bit_exact(beta, dtype, kind):
    V = 151936 if dtype == "bf16" else 50000
    cfg = synth.get_config("qwen3_8b").with_(batch=4, branch=beta, vocab=V)
    taus = []
    for seed in range(3):
        topk = synth.make_random_topk(cfg, seed=seed)
        tree = oracle.build_tree(topk, np.arange(4, dtype=np.int32), np.full(4, 9, np.int32))
        lg = synth.make_target_logits(cfg, tree["node_token"], tree["node_parent"], seed=seed, kind=kind,
                                      dtype=dtype)
        if seed == 1:  # planted exact ties of the maximum: the smaller id must win
            for b in range(4):
                m = int(tree["node_token"][b, 1]) if beta > 0 else 0
                row = lg[b, 0]
                mx = row.max()
                row[m] = mx
                row[(m + 17) % V] = mx
                row[5] = np.nan
                # every other row (leaves included, whose argmax the walk scans itself) gets a
                # second copy of its maximum
                for node in range(1, lg.shape[1]):
                    r2 = lg[b, node]
                    k = int(np.nanargmax(r2))
                    r2[(k + 17) % V] = r2[k]
        t_dt = torch.bfloat16 if dtype == "bf16" else torch.float32
        lt = torch.from_numpy(lg).to("cuda:0").to(t_dt)
        got = _accept_gpu(tree["node_token"], tree["node_parent"], lt, cfg.block)
        want = oracle.verify_accept(tree["node_token"], tree["node_parent"], lg, cfg.block)
        for k in want:
            np.testing.assert_array_equal(got[k], want[k], err_msg=f"{k} seed={seed}")
        taus += list(want["accept_len"] + 1)
    log(f"tau values: {taus}")


def test_verify_accept_bad_tree_sets_error_word_then_clears():
    """A parent that does not precede its node raises DEV_BAD_TREE (the walk
    still ends); the next call on the same workspace starts from a clear error
    word and matches the oracle."""
    from paper_2605_29707_amd import binding as bd
    V = 5000
    cfg = synth.get_config("qwen3_8b").with_(batch=2, branch=2, vocab=V)
    topk = synth.make_random_topk(cfg, seed=7)
    tree = oracle.build_tree(topk, np.arange(2, dtype=np.int32), np.full(2, 9, np.int32))
    lg = synth.make_target_logits(cfg, tree["node_token"], tree["node_parent"], seed=7, dtype="f32")
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bs, nn = tree["node_token"].shape
    acc = torch.empty(bs, dtype=torch.int32, device=dev)
    nodes = torch.empty(bs, cfg.block - 1, dtype=torch.int32, device=dev)
    out = torch.empty(bs, cfg.block, dtype=torch.int32, device=dev)
    ws = torch.empty(bd.domino_verify_workspace_bytes(bs, nn, V), dtype=torch.uint8, device=dev)
    bad = tree["node_parent"].copy()
    bad[1, 3] = 7
    bd.domino_verify_accept(t(tree["node_token"]), t(bad), t(lg), cfg.block, acc, nodes, out, ws)
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(ws) & bd.DEV_BAD_TREE
    bd.domino_verify_accept(t(tree["node_token"]), t(tree["node_parent"]), t(lg), cfg.block, acc, nodes, out, ws)
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(ws) == 0
    want = oracle.verify_accept(tree["node_token"], tree["node_parent"], lg, cfg.block)
    np.testing.assert_array_equal(acc.cpu().numpy(), want["accept_len"])
    np.testing.assert_array_equal(nodes.cpu().numpy(), want["accepted_nodes"])
    np.testing.assert_array_equal(out.cpu().numpy(), want["out_tokens"])


def test_tiny_pipeline_draft_tree_accept():
    cfg = synth.get_config("tiny").with_(ctx_from_hidden=False, batch=2, branch=4)
    w = synth.make_weights(cfg, seed=7)
    inp = synth.make_inputs(cfg, seed=7)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=4)
    g = run.step(inp)
    tree_g = _tree_gpu(g["topk_ids"], inp["anchor"], inp["ctx_lens"])
    tree_o = oracle.build_tree(g["topk_ids"], inp["anchor"], inp["ctx_lens"])
    for k in tree_o:
        np.testing.assert_array_equal(tree_g[k], tree_o[k])
    lg = synth.make_target_logits(cfg, tree_o["node_token"], tree_o["node_parent"], seed=7, dtype="f32")
    got = _accept_gpu(tree_g["node_token"], tree_g["node_parent"], torch.from_numpy(lg).cuda(), cfg.block)
    want = oracle.verify_accept(tree_o["node_token"], tree_o["node_parent"], lg, cfg.block)
    for k in want:
        np.testing.assert_array_equal(got[k], want[k])
    run.close()


# ---------------------------------------------------------------- full size
def test_qwen3_8b_bs1_full_size_parity():
    """The benchmarked workload: Qwen3-8B shape, bs 1, ctx 1024, k = 16, bf16."""
    cfg = synth.get_config("qwen3_8b")
    log("generating qwen3_8b weights")
    w = synth.make_weights(cfg, seed=0)
    inp = synth.make_inputs(cfg, seed=0)
    log("uploading + packing")
    from paper_2605_29707_amd import binding as bd
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    plain = run.step(inp, debug=False)
    log("gpu step done")
    assert bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    gpu = run.step(inp, debug=True)
    np.testing.assert_array_equal(plain["topk_ids"], gpu["topk_ids"])
    np.testing.assert_array_equal(plain["topk_vals"], gpu["topk_vals"])
    assert gpu["err"] == 0
    run.close()
    del run
    torch.cuda.empty_cache()
    log("oracle (fp64)")
    w64 = oracle.as_f64_weights(w)
    del w
    ref = oracle_for(cfg, w64, inp, gpu, 1)
    log("comparing")
    n = check_against_oracle(cfg, gpu, ref, 2e-2, 1)
    log(f"top-1 positions checked: {n}")
    assert n >= 12


def persistent_config(batch):
    """The tiny drafter with d_s = 256 and a 8192-token vocabulary, bf16: the
    persistent rollout takes it (13 workgroups of 640 vocabulary rows, whose
    share of the 1024 rows of [W1 S-half; W_hh] fits in LDS; at d_s = 1024 and
    4096 tokens its 7 workgroups could not hold theirs, and the launch-pair
    rollout runs)."""
    return synth.get_config("tiny").with_(dtype="bf16", batch=batch, gru_hidden=256, vocab=8192,
                                          ctx_from_hidden=False)


@pytest.mark.parametrize("batch", [1, 2, 3, 4])
def test_persistent_rollout_matches_launch_pair_rollout(batch, monkeypatch):
    """bf16, r = 256, one to four batch rows, greedy: the rollout runs as one
    persistent launch per pair of rows (an ordinary launch after an occupancy
    check) with the W2 slice held on chip.  It must agree with the launch-pair rollout
    (DOMINO_ROLLOUT=loop at model creation): the backbone outputs bit for bit,
    states and logits to fp32 summation order, the drafted tokens exactly away
    from near-ties; free-running and teacher-forced.  Each run checks which
    rollout path its steps took, so neither side can silently be the other."""
    from paper_2605_29707_amd import binding as bd
    cfg = persistent_config(batch)
    w = synth.make_weights(cfg, seed=21, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=21)
    f = synth.make_forced_tokens(cfg, seed=21)
    monkeypatch.delenv("DOMINO_ROLLOUT", raising=False)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    a = run.step(inp)
    assert bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    af = run.step(inp, forced=f)
    assert bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    run.close()
    monkeypatch.setenv("DOMINO_ROLLOUT", "loop")
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    b = run.step(inp)
    assert not bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    bf = run.step(inp, forced=f)
    assert not bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    run.close()
    for x, y, forced in ((a, b, False), (af, bf, True)):
        assert x["err"] == 0 and y["err"] == 0
        for k in ("hidden", "base_logits"):
            np.testing.assert_array_equal(x[k], y[k], err_msg=k)
        # a free-running rollout follows its own tokens: positions after the first
        # differing token (a near-tie, which must be one) are not comparable
        upto = np.full(batch, cfg.depth)
        if not forced:
            for r in range(batch):
                diff = np.nonzero(x["topk_ids"][r, :, 0] != y["topk_ids"][r, :, 0])[0]
                if diff.size:
                    j = diff[0]
                    s = np.sort(y["final_logits"][r, j])
                    assert s[-1] - s[-2] < 1e-3, (r, j)
                    upto[r] = j + 1
        for r in range(batch):
            n = upto[r]
            es = float(np.abs(x["states"][r, :n] - y["states"][r, :n]).max())
            el = float(np.abs(x["final_logits"][r, :n] - y["final_logits"][r, :n]).max())
            log(f"persistent vs launch-pair ({'forced' if forced else 'free'}, row {r}, {n} positions): "
                f"states within {es:.2e}, final logits within {el:.2e}")
            assert es < 1e-5 and el < 1e-4
            np.testing.assert_allclose(x["topk_vals"][r, :n], y["topk_vals"][r, :n], atol=1e-4, rtol=0)
    ref = oracle_for(cfg, oracle.as_f64_weights(w), inp, a, 1)
    check_against_oracle(cfg, a, ref, 2e-2, 1)


def test_persistent_rollout_wait_gives_up_then_recovers():
    """The failure path of the persistent rollout, forced from the host: with a
    poll limit of 0 every wait gives up at once, raises DEV_BARRIER_TIMEOUT and
    every workgroup leaves (the launch ends); with
    the default restored, the next step on the same workspace is clean and
    matches a run that never failed."""
    from paper_2605_29707_amd import binding as bd
    cfg = persistent_config(1)
    w = synth.make_weights(cfg, seed=22, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=22)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    good = run.step(inp)
    assert good["err"] == 0
    assert bd.domino_debug_last_paths(run.model) & bd.PATH_PERSISTENT_ROLLOUT
    bd.domino_debug_set_poll_limit(run.model, 0)
    bad = run.step(inp)
    log(f"forced timeout: error word {bad['err']:#x}")
    assert bad["err"] & bd.DEV_BARRIER_TIMEOUT
    bd.domino_debug_set_poll_limit(run.model, -1)
    again = run.step(inp)
    run.close()
    assert again["err"] == 0
    for k in ("topk_ids", "topk_vals", "final_logits", "states"):
        np.testing.assert_array_equal(again[k], good[k], err_msg=k)

