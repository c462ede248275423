"""Pins for the training-forward oracle (teacher-forced forward and the
base-anchored curriculum loss), on the CPU: closed forms of the cross-entropy,
torch's fp64 cross_entropy, the curriculum's end points, and the zero-head
case where final and base logits coincide."""
import numpy as np
import pytest

import oracle
import synth

to = oracle.train_oracle


def test_cross_entropy_closed_forms():
    assert to.cross_entropy(np.zeros(37), 5) == pytest.approx(np.log(37), abs=1e-12)
    z = np.array([2.0, 0.0, -1.0])
    assert to.cross_entropy(z, 0) == pytest.approx(-np.log(np.exp(2) / np.sum(np.exp(z))), abs=1e-12)
    assert to.cross_entropy(np.array([0.0, np.nan, 0.0]), 2) == pytest.approx(np.log(2), abs=1e-12)


def test_cross_entropy_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    z = rng.normal(size=(6, 300)) * 3
    lab = rng.integers(0, 300, size=6)
    want = torch.nn.functional.cross_entropy(torch.from_numpy(z), torch.from_numpy(lab), reduction="none").numpy()
    got = np.array([to.cross_entropy(z[i], lab[i]) for i in range(6)])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_position_weights():
    w = to.position_weights(15, 7.0)
    assert w[0] == 1.0
    np.testing.assert_allclose(w[1:] / w[:-1], np.exp(-1 / 7.0), rtol=1e-14)
    assert np.all(to.position_weights(5, 1e12) > 1 - 1e-10)     # gamma -> inf: unweighted


def test_curriculum_end_points_and_weighted_mean():
    rng = np.random.default_rng(1)
    bs, depth, V = 3, 15, 50
    base = rng.normal(size=(bs, depth, V))
    final = base + rng.normal(size=(bs, depth, V))
    lab = rng.integers(0, V, size=(bs, depth))
    tot1, lb, lf, ce_b, ce_f = to.curriculum_loss(base, final, lab, 1.0, 15.0)
    tot0, _, _, _, _ = to.curriculum_loss(base, final, lab, 0.0, 15.0)
    assert tot1 == pytest.approx(lb, abs=1e-12) and tot0 == pytest.approx(lf, abs=1e-12)
    tot, _, _, _, _ = to.curriculum_loss(base, final, lab, 0.3, 15.0)
    assert tot == pytest.approx(0.7 * lf + 0.3 * lb, abs=1e-12)
    w = to.position_weights(depth, 15.0)
    assert lb == pytest.approx(float(np.sum(ce_b * w) / (bs * np.sum(w))), abs=1e-12)
    # a single position carrying all the loss
    ce_one = np.zeros((bs, depth)); ce_one[:, 4] = 2.0
    assert float(np.sum(ce_one * w) / (bs * np.sum(w))) == pytest.approx(2.0 * w[4] / np.sum(w))


def test_zero_head_final_equals_base():
    cfg = synth.get_config("tiny").with_(batch=2)
    w = synth.make_weights(cfg, seed=3, zero_head=True)
    inp = synth.make_inputs(cfg, seed=3)
    lab = synth.make_forced_tokens(cfg, seed=3)
    ref = to.train_forward(cfg, oracle.as_f64_weights(w), inp["anchor"], inp["ctx_lens"], inp["ctx_k"],
                           inp["ctx_v"], lab, 0.4, 15.0, ctx_hidden=inp["ctx_hidden"])
    assert ref["loss_final"] == pytest.approx(ref["loss_base"], abs=1e-12)
    assert ref["loss"] == pytest.approx(ref["loss_base"], abs=1e-12)


def test_labels_align_with_draft_positions():
    """Labels set to the free greedy rollout's own tokens: the teacher-forced
    forward reproduces that rollout exactly, and at every position the label
    is the final logits' argmax, so its cross-entropy is the smallest any
    label could get (a label paired with the wrong position fails this)."""
    cfg = synth.get_config("tiny").with_(batch=2)
    w = oracle.as_f64_weights(synth.make_weights(cfg, seed=4, gain_std=0.1))
    inp = synth.make_inputs(cfg, seed=4)
    args = (inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"])
    free = oracle.draft_step(cfg, w, *args, 1, ctx_hidden=inp["ctx_hidden"])
    lab = free["topk_ids"][:, :, 0]
    ref = to.train_forward(cfg, w, *args, lab, 0.5, 15.0, ctx_hidden=inp["ctx_hidden"])
    np.testing.assert_array_equal(ref["final_logits"], free["final_logits"])
    for b in range(cfg.batch):
        for k in range(cfg.depth):
            z = ref["final_logits"][b, k]
            lse = np.log(np.sum(np.exp(z - z.max()))) + z.max()
            assert ref["ce_final"][b, k] == pytest.approx(lse - z.max(), abs=1e-9)
            other = (lab[b, k] + 1) % cfg.vocab
            assert ref["ce_final"][b, k] <= to.cross_entropy(z, other)
