"""C-ABI checks that need no GPU: the library loads, exports every function
include/domino.h declares, and rejects invalid arguments before any HIP call."""
import ctypes as C
import os
import re

import pytest

from paper_2605_29707_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "domino.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(domino_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = bd.load()
    names = header_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(bd.exported_symbols()) == names


def _cfg(**kw):
    c = dict(hidden=256, n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=1024, vocab=4096,
             block=16, gru_hidden=1024, rank=256, mask_token_id=4095, rms_eps=1e-6, rope_theta=1e6,
             dtype=bd.DOMINO_F32)
    c.update(kw)
    return bd.domino_config(**c)


@pytest.mark.parametrize("kw,status", [
    ({"hidden": 0}, bd.DOMINO_ERR_INVALID_ARG),
    ({"block": 1}, bd.DOMINO_ERR_INVALID_ARG),
    ({"block": 65}, bd.DOMINO_ERR_INVALID_ARG),
    ({"mask_token_id": 4096}, bd.DOMINO_ERR_INVALID_ARG),
    ({"dtype": 7}, bd.DOMINO_ERR_INVALID_ARG),
    ({"head_dim": 96}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"n_kv_heads": 3}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"hidden": 250}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"rank": 1000}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"rank": 64}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"gru_hidden": 2048}, bd.DOMINO_ERR_UNSUPPORTED),
    ({"ctx_fuse_layers": -1}, bd.DOMINO_ERR_INVALID_ARG),
    ({"ctx_fuse_layers": 9}, bd.DOMINO_ERR_INVALID_ARG),
    ({}, bd.DOMINO_ERR_INVALID_ARG),  # valid config, NULL weights
])
def test_model_create_validation(kw, status):
    lib = bd.load()
    h = C.c_void_p()
    cfg = _cfg(**kw)
    assert lib.domino_model_create(C.byref(cfg), None, C.byref(h)) == status
    assert h.value is None
    assert bd.last_error()


def test_context_fusion_needs_its_weight():
    # every pointer set (never dereferenced: validation precedes any HIP call)
    # except ctx_fc, which a config with fused context layers requires
    lib = bd.load()
    fake = 4096
    arr = (C.c_void_p * 2)(fake, fake)
    pp = C.cast(arr, C.POINTER(C.c_void_p))
    w = bd.domino_weights(embed=fake, lm_head=fake, final_norm=fake,
                          **{k: pp for k in ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo",
                                             "ffn_norm", "w_gate", "w_up", "w_down")},
                          **{k: fake for k in ("gru_w_ih", "gru_w_hh", "gru_b_ih", "gru_b_hh", "w1", "w2")},
                          ctx_fc=None)
    h = C.c_void_p()
    cfg = _cfg(ctx_fuse_layers=3)
    assert lib.domino_model_create(C.byref(cfg), C.byref(w), C.byref(h)) == bd.DOMINO_ERR_INVALID_ARG
    assert h.value is None and "ctx_fc" in bd.last_error()


def test_null_config_and_out():
    lib = bd.load()
    h = C.c_void_p()
    assert lib.domino_model_create(None, None, C.byref(h)) == bd.DOMINO_ERR_INVALID_ARG
    cfg = _cfg()
    assert lib.domino_model_create(C.byref(cfg), None, None) == bd.DOMINO_ERR_INVALID_ARG


def test_draft_step_validation_without_model():
    lib = bd.load()
    st = lib.domino_draft_step(None, 1, None, None, None, None, 0, None, 0, 1, None, None, None, None,
                               None, 0, None)
    assert st == bd.DOMINO_ERR_INVALID_ARG
    assert "model" in bd.last_error()
    assert lib.domino_workspace_bytes(None, 1, 16, 0, 1) == 0


def test_tree_and_accept_validation():
    lib = bd.load()
    p = C.c_void_p(16)  # never dereferenced: validation fails first
    assert lib.domino_build_tree(0, 15, 1, p, p, p, p, p, p, p, None, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_build_tree(1, 0, 1, p, p, p, p, p, p, p, None, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_build_tree(1, 15, 9, p, p, p, p, p, p, p, None, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_build_tree(1, 15, 1, None, p, p, p, p, p, p, None, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_workspace_bytes(1, 0, 10) == 0
    assert lib.domino_verify_workspace_bytes(1, 2000, 10) == 0
    assert lib.domino_verify_workspace_bytes(2, 16, 151936) > 0
    args = (1, 16, 100, 16, p, p, p, bd.DOMINO_F32, p, p, p)
    assert lib.domino_verify_accept(*args, None, 10**9, None) == bd.DOMINO_ERR_WORKSPACE
    assert lib.domino_verify_accept(*args, p, 1, None) == bd.DOMINO_ERR_WORKSPACE
    assert lib.domino_verify_accept(1, 16, 100, 1, p, p, p, bd.DOMINO_F32, p, p, p, p, 10**9, None) == \
        bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_accept(1, 16, 100, 16, p, p, p, 5, p, p, p, p, 10**9, None) == \
        bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_workspace_error(None, None, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_profile_enable(None, 1) == bd.DOMINO_ERR_INVALID_ARG


def test_sampling_entry_points_validation():
    lib = bd.load()
    p = C.c_void_p(16)  # never dereferenced: validation fails first
    # sampled drafting: model, temperature and the required final_logits are checked first
    st = lib.domino_draft_step_sampled(None, 1, p, p, p, p, 16, None, 0, 1.0, 7, None, p, p, p, None, p, 10**9,
                                       None)
    assert st == bd.DOMINO_ERR_INVALID_ARG
    for t in (0.0, -1.0, float("inf"), float("nan")):
        st = lib.domino_draft_step_sampled(None, 1, p, p, p, p, 16, None, 0, t, 7, None, p, p, p, None, p, 10**9,
                                           None)
        assert st == bd.DOMINO_ERR_INVALID_ARG and "temperature" in bd.last_error()
    st = lib.domino_draft_step_sampled(None, 1, p, p, p, p, 16, None, 0, 1.0, 7, None, p, p, None, None, p,
                                       10**9, None)
    assert st == bd.DOMINO_ERR_INVALID_ARG and "final_logits" in bd.last_error()
    # sampled verification
    assert lib.domino_verify_sample_workspace_bytes(1, 1, 100) == 0
    assert lib.domino_verify_sample_workspace_bytes(1, 16, 0) == 0
    assert lib.domino_verify_sample_workspace_bytes(2, 16, 151936) > 0
    ok = (1, 16, 100, p, p, bd.DOMINO_BF16, p)
    assert lib.domino_verify_sample(*ok, 0.0, 1, p, p, p, p, 10**9, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_sample(1, 1, 100, p, p, bd.DOMINO_F32, p, 1.0, 1, p, p, p, p, 10**9, None) == \
        bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_sample(1, 16, 100, p, p, 9, p, 1.0, 1, p, p, p, p, 10**9, None) == \
        bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_sample(*ok, 1.0, 1, p, p, None, p, 10**9, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_verify_sample(*ok, 1.0, 1, p, p, p, None, 10**9, None) == bd.DOMINO_ERR_WORKSPACE
    assert lib.domino_verify_sample(*ok, 1.0, 1, p, p, p, p, 8, None) == bd.DOMINO_ERR_WORKSPACE
    assert lib.domino_philox4x32_10(None, 0, None, 4, None) == bd.DOMINO_ERR_INVALID_ARG
    assert lib.domino_philox4x32_10(None, 0, None, -1, None) == bd.DOMINO_ERR_INVALID_ARG


def test_train_entry_points_validation():
    lib = bd.load()
    p = C.c_void_p(16)  # never dereferenced: validation fails first
    assert lib.domino_train_workspace_bytes(None, 1, 16, 0) == 0
    base = (None, 1, p, p, p, p, 16, None, 0)
    st = lib.domino_train_forward(*base, p, 0.5, 15.0, p, None, None, p, 10**9, None)
    assert st == bd.DOMINO_ERR_INVALID_ARG and "model" in bd.last_error()


def test_target_entry_points_validation():
    lib = bd.load()
    p = C.c_void_p(16)  # never dereferenced: validation fails first
    h = C.c_void_p()
    cfg = _cfg(gru_hidden=0, rank=0)        # head sizes are ignored for a target decoder
    assert lib.domino_target_create(C.byref(cfg), None, C.byref(h)) == bd.DOMINO_ERR_INVALID_ARG
    assert "weights" in bd.last_error() and h.value is None
    cfg = _cfg(head_dim=96)
    assert lib.domino_target_create(C.byref(cfg), None, C.byref(h)) == bd.DOMINO_ERR_UNSUPPORTED
    assert lib.domino_target_workspace_bytes(None, 1, 16, 1024) == 0
    st = lib.domino_target_verify(None, 1, 16, p, p, p, p, p, p, 1024, p, bd.DOMINO_BF16, p, 10**9, None)
    assert st == bd.DOMINO_ERR_INVALID_ARG and "model" in bd.last_error()
    st = lib.domino_target_commit(None, 1, 16, 15, p, p, p, p, p, 1024, p, p, None)
    assert st == bd.DOMINO_ERR_INVALID_ARG


def test_appended_rows_must_match_the_context_width():
    # host-side check before any launch: fused configs take k*d-wide fp32 rows
    import types
    import torch
    cfg = types.SimpleNamespace(hidden=64, ctx_fuse_layers=3)
    model = types.SimpleNamespace(cfg=cfg)
    ok = torch.zeros(2, 5, 192, dtype=torch.float32)
    bd._check_ctx_hidden(model, 2, ok, 5)
    bd._check_ctx_hidden(model, 2, None, 0)
    for bad in (torch.zeros(2, 5, 64, dtype=torch.float32),      # d-wide rows for a fused config
                torch.zeros(2, 5, 192, dtype=torch.float64),     # wrong dtype
                torch.zeros(2, 192, 5, dtype=torch.float32).transpose(1, 2)):  # not contiguous
        with pytest.raises(bd.DominoError):
            bd._check_ctx_hidden(model, 2, bad, 5)
    cfg0 = types.SimpleNamespace(hidden=64, ctx_fuse_layers=0)
    bd._check_ctx_hidden(types.SimpleNamespace(cfg=cfg0), 2, torch.zeros(2, 5, 64), 5)


def test_noalloc_accept_rejects_sizes_beyond_its_scratch():
    """domino_verify_accept_noalloc checks the argmax partials against its fixed
    scratch before any HIP call: 64 rows x 1024 nodes x 38 vocabulary chunks x 8
    bytes (19.9 MB) exceed DOMINO_NOALLOC_SCRATCH_BYTES."""
    lib = bd.load()
    p = 16  # never dereferenced: the size check comes first
    st = lib.domino_verify_accept_noalloc(64, 1024, 151936, 16, p, p, p, bd.DOMINO_BF16, p, p, p, p, None)
    assert st == bd.DOMINO_ERR_UNSUPPORTED
    assert "scratch" in bd.last_error()
    assert lib.domino_verify_accept_noalloc(1, 16, 100, 16, p, p, p, bd.DOMINO_F32, p, p, p, None, None) == \
        bd.DOMINO_ERR_INVALID_ARG
