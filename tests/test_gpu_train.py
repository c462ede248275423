"""GPU parity of the teacher-forced training forward and curriculum loss
(Sec. 4.2) through the C-ABI, against the training oracle.

Compared: the hidden states, base and final logits, GRU states, the
per-position cross-entropies and the three losses.  Logits keep the drafting
bar (1e-4 absolute fp32, 2e-2 bf16).  A cross-entropy is a log-sum-exp minus
one logit, each within the logit error of the oracle's, and the losses are
weighted means of cross-entropies, so both are held to twice the logit bar.
The forward must also agree with the draft step teacher-forced on the same
labels: bit for bit on the hidden states, base logits and GRU states (the same
kernels), and to fp32 rounding on the final logits (u comes from one batched
matrix-core product there instead of per-position dot products).
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import GpuRun, log

to = oracle.train_oracle
pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_29707_amd import binding as bd  # noqa: E402

GAMMA = 15.0


def _train(run, inp, labels, lam, gamma=GAMMA, debug=True, ctx_lens=None):
    cfg = run.cfg
    bs, D, V = cfg.batch, cfg.depth, cfg.vocab
    dev = run.dev
    ws = torch.empty(bd.domino_train_workspace_bytes(run.model, bs, run.max_ctx, run.n_new), dtype=torch.uint8,
                     device=dev)
    loss = torch.empty(3, dtype=torch.float32, device=dev)
    ce = torch.empty(2, bs, D, dtype=torch.float32, device=dev)
    dbg = None
    if debug:
        dbg = {"hidden": torch.empty(bs, D, cfg.hidden, device=dev),
               "base_logits": torch.empty(bs, D, V, device=dev),
               "final_logits": torch.empty(bs, D, V, device=dev),
               "states": torch.empty(bs, D, cfg.gru_hidden, device=dev)}
    hid = run.t(inp["ctx_hidden"]) if run.n_new > 0 else None
    bd.domino_train_forward(run.model, run.t(inp["anchor"], torch.int32),
                            run.t(inp["ctx_lens"] if ctx_lens is None else ctx_lens, torch.int32),
                            run.t(inp["ctx_k"], run.kv_dtype()), run.t(inp["ctx_v"], run.kv_dtype()), run.max_ctx,
                            run.t(labels, torch.int32), lam, gamma, loss, ws, ce=ce, ctx_hidden_new=hid,
                            n_new=run.n_new, debug=dbg)
    torch.cuda.synchronize()
    out = {"loss": loss.cpu().numpy(), "ce": ce.cpu().numpy(), "err": bd.domino_workspace_error(ws)}
    if debug:
        out.update({k: v.cpu().numpy() for k, v in dbg.items()})
    return out


def _check(gpu, ref, tol):
    errs = {k: float(np.abs(gpu[k] - ref[k]).max()) for k in ("hidden", "base_logits", "final_logits", "states")}
    errs["ce_base"] = float(np.abs(gpu["ce"][0] - ref["ce_base"]).max())
    errs["ce_final"] = float(np.abs(gpu["ce"][1] - ref["ce_final"]).max())
    want = np.array([ref["loss"], ref["loss_base"], ref["loss_final"]])
    errs["loss"] = float(np.abs(gpu["loss"] - want).max())
    log("max |gpu - oracle|: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    log(f"losses gpu {gpu['loss'].tolist()} oracle {want.tolist()}")
    for k, v in errs.items():
        assert v < (2 * tol if k.startswith(("ce", "loss")) else tol), (k, v)


def test_train_tiny_f32_context_from_hidden_states():
    cfg = synth.get_config("tiny").with_(batch=2)
    w = synth.make_weights(cfg, seed=11, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=11)
    labels = synth.make_forced_tokens(cfg, seed=11)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1, n_new=inp["ctx_hidden"].shape[1])
    gpu = _train(run, inp, labels, 0.3)
    run.close()
    assert gpu["err"] == 0
    ref = to.train_forward(cfg, oracle.as_f64_weights(w), inp["anchor"], inp["ctx_lens"], inp["ctx_k"],
                           inp["ctx_v"], labels, 0.3, GAMMA, ctx_hidden=inp["ctx_hidden"])
    _check(gpu, ref, 1e-4)


@pytest.mark.parametrize("batch,lens", [(5, [128, 37, 0, 90, 1]), (12, [(41 * i) % 129 for i in range(12)])])
def test_train_tiny_bf16_ragged(batch, lens):
    """batch 5 runs the fused state kernel, batch 12 the separate gru and u kernels."""
    cfg = synth.get_config("tiny").with_(dtype="bf16", batch=batch, ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=12, gain_std=0.1)
    lens = np.array(lens, np.int32)
    inp = synth.make_inputs(cfg, seed=12, ctx_lens=lens, max_ctx=128)
    labels = synth.make_forced_tokens(cfg, seed=12)
    run = GpuRun(cfg, w, 128, beta=1)
    gpu = _train(run, inp, labels, 0.7)
    run.close()
    assert gpu["err"] == 0
    ref = to.train_forward(cfg, oracle.as_f64_weights(w), inp["anchor"], lens, inp["ctx_k"], inp["ctx_v"], labels,
                           0.7, GAMMA)
    _check(gpu, ref, 2e-2)


def test_train_matches_teacher_forced_draft_step():
    cfg = synth.get_config("tiny").with_(dtype="bf16", batch=3, ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=13, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=13)
    labels = synth.make_forced_tokens(cfg, seed=13)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    gpu = _train(run, inp, labels, 0.5)
    drf = run.step(inp, forced=labels)
    run.close()
    for k in ("hidden", "base_logits", "states"):
        np.testing.assert_array_equal(gpu[k], drf[k], err_msg=k)
    err = float(np.abs(gpu["final_logits"] - drf["final_logits"]).max())
    log(f"training forward vs teacher-forced draft step: final logits within {err:.2e}, the rest bit-identical")
    assert err < 1e-5


def test_train_curriculum_end_points_determinism_and_bad_label():
    cfg = synth.get_config("tiny").with_(dtype="bf16", batch=4, ctx_from_hidden=False)
    w = synth.make_weights(cfg, seed=14, gain_std=0.1)
    inp = synth.make_inputs(cfg, seed=14)
    labels = synth.make_forced_tokens(cfg, seed=14)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    a = _train(run, inp, labels, 1.0, debug=False)
    b = _train(run, inp, labels, 1.0, debug=True)
    c = _train(run, inp, labels, 0.0, debug=False)
    # debug stores change nothing, and repeated runs are bit-identical
    np.testing.assert_array_equal(a["loss"], b["loss"])
    np.testing.assert_array_equal(a["ce"], b["ce"])
    assert a["loss"][0] == a["loss"][1] and c["loss"][0] == c["loss"][2]
    np.testing.assert_array_equal(a["loss"][1:], c["loss"][1:])
    # the last label never reaches the encoder; it must still be range-checked
    bad = labels.copy()
    bad[2, cfg.depth - 1] = cfg.vocab
    d = _train(run, inp, bad, 0.5, debug=False)
    run.close()
    assert d["err"] & bd.DEV_BAD_TOKEN
    assert np.isnan(d["ce"][:, 2, cfg.depth - 1]).all()
    mask = np.ones((cfg.batch, cfg.depth), bool)
    mask[2, cfg.depth - 1] = False
    np.testing.assert_array_equal(d["ce"][:, mask], a["ce"][:, mask])
    assert np.isnan(d["loss"]).all()


def test_train_qwen3_8b_full_size():
    cfg = synth.get_config("qwen3_8b")
    w = synth.make_weights(cfg, seed=0)
    inp = synth.make_inputs(cfg, seed=0)
    labels = synth.make_forced_tokens(cfg, seed=0)
    run = GpuRun(cfg, w, inp["max_ctx"], beta=1)
    plain = _train(run, inp, labels, 0.5, debug=False)   # the benchmark's configuration
    gpu = _train(run, inp, labels, 0.5, debug=True)
    run.close()
    del run
    torch.cuda.empty_cache()
    assert gpu["err"] == 0
    np.testing.assert_array_equal(plain["loss"], gpu["loss"])
    w64 = oracle.as_f64_weights(w, keep=("embed",))
    del w
    ref = to.train_forward(cfg, w64, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], labels, 0.5, GAMMA)
    _check(gpu, ref, 2e-2)
