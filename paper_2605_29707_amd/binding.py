"""ctypes binding of libdomino.so (include/domino.h), argument marshalling only.

Every function here forwards to the C entry point of the same name; torch is
used only to hold device memory and to name streams.  The library must have
been built (paper_2605_29707_amd/build.py); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdomino.so")

DOMINO_OK = 0
DOMINO_ERR_INVALID_ARG = -1
DOMINO_ERR_WORKSPACE = -2
DOMINO_ERR_UNSUPPORTED = -3
DOMINO_ERR_HIP = -4
DOMINO_ERR_DEVICE = -5
DOMINO_F32, DOMINO_BF16 = 0, 1

DEV_BAD_TOKEN, DEV_BAD_CTX_LEN, DEV_BAD_TREE, DEV_BARRIER_TIMEOUT = 1, 2, 4, 8

KERNEL_CLASSES = ["embed", "norm", "qkv", "rope", "attn", "wo", "gateup", "down", "lmhead", "w1h",
                  "headloop", "ctxproj", "trainloss"]


class domino_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "hidden", "n_layers", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "vocab",
        "block", "gru_hidden", "rank", "mask_token_id")] + [
        ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("dtype", C.c_int),
        ("ctx_fuse_layers", C.c_int32)]


_VP = C.c_void_p
_PP = C.POINTER(C.c_void_p)


class domino_weights(C.Structure):
    _fields_ = [("embed", _VP), ("lm_head", _VP), ("final_norm", _VP)] + [
        (n, _PP) for n in ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo", "ffn_norm",
                           "w_gate", "w_up", "w_down")] + [
        (n, _VP) for n in ("gru_w_ih", "gru_w_hh", "gru_b_ih", "gru_b_hh", "w1", "w2", "ctx_fc")]


class domino_debug(C.Structure):
    _fields_ = [(n, _VP) for n in ("hidden", "base_logits", "final_logits", "states")]


class DominoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"domino status {status}: {msg}")
        self.status = status


_lib = None


def load() -> C.CDLL:
    """Load libdomino.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2605_29707_amd/build.py")
    lib = C.CDLL(LIB_PATH)
    i32, sz, u32 = C.c_int32, C.c_size_t, C.c_uint32
    P = C.c_void_p
    sig = {
        "domino_model_create": (i32, [C.POINTER(domino_config), C.POINTER(domino_weights), C.POINTER(P)]),
        "domino_model_destroy": (None, [P]),
        "domino_workspace_bytes": (sz, [P, i32, i32, i32, i32]),
        "domino_last_error": (C.c_char_p, []),
        "domino_draft_step": (i32, [P, i32, P, P, P, P, i32, P, i32, i32, P, P, P,
                                    C.POINTER(domino_debug), P, sz, P]),
        "domino_build_tree": (i32, [i32, i32, i32, P, P, P, P, P, P, P, P, P]),
        "domino_verify_workspace_bytes": (sz, [i32, i32, i32]),
        "domino_verify_accept": (i32, [i32, i32, i32, i32, P, P, P, C.c_int, P, P, P, P, sz, P]),
        "domino_workspace_error": (i32, [P, P, C.POINTER(i32)]),
        "domino_workspace_clear_error": (i32, [P, P]),
        "domino_profile_enable": (i32, [P, u32]),
        "domino_profile_read": (i32, [P, i32, C.POINTER(C.c_double), C.POINTER(i32)]),
        "domino_profile_reset": (i32, [P]),
        "domino_debug_set_poll_limit": (i32, [P, i32]),
        "domino_debug_last_paths": (i32, [P, C.POINTER(u32)]),
        "domino_verify_accept_noalloc": (i32, [i32, i32, i32, i32, P, P, P, C.c_int, P, P, P, P, P]),
        "domino_draft_step_sampled": (i32, [P, i32, P, P, P, P, i32, P, i32, C.c_float, C.c_uint64, P, P, P, P,
                                            C.POINTER(domino_debug), P, sz, P]),
        "domino_verify_sample_workspace_bytes": (sz, [i32, i32, i32]),
        "domino_verify_sample": (i32, [i32, i32, i32, P, P, C.c_int, P, C.c_float, C.c_uint64, P, P, P, P, sz,
                                       P]),
        "domino_philox4x32_10": (i32, [P, C.c_uint64, P, i32, P]),
        "domino_train_workspace_bytes": (sz, [P, i32, i32, i32]),
        "domino_target_create": (i32, [C.POINTER(domino_config), C.POINTER(domino_weights), C.POINTER(P)]),
        "domino_target_workspace_bytes": (sz, [P, i32, i32, i32]),
        "domino_target_verify": (i32, [P, i32, i32, P, P, P, P, P, P, i32, P, C.c_int, P, sz, P]),
        "domino_target_commit": (i32, [P, i32, i32, i32, P, P, P, P, P, i32, P, P, P]),
        "domino_train_forward": (i32, [P, i32, P, P, P, P, i32, P, i32, P, C.c_float, C.c_float, P, P,
                                       C.POINTER(domino_debug), P, sz, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def exported_symbols():
    return ["domino_model_create", "domino_model_destroy", "domino_workspace_bytes", "domino_last_error",
            "domino_draft_step", "domino_build_tree", "domino_verify_workspace_bytes",
            "domino_verify_accept", "domino_workspace_error", "domino_workspace_clear_error",
            "domino_profile_enable", "domino_profile_read", "domino_profile_reset",
            "domino_draft_step_sampled", "domino_verify_sample_workspace_bytes", "domino_verify_sample",
            "domino_philox4x32_10", "domino_train_workspace_bytes", "domino_train_forward",
            "domino_target_create", "domino_target_workspace_bytes", "domino_target_verify", "domino_target_commit",
            "domino_debug_set_poll_limit", "domino_debug_last_paths", "domino_verify_accept_noalloc"]


def last_error() -> str:
    return load().domino_last_error().decode()


def _check(status: int):
    if status != DOMINO_OK:
        raise DominoError(status, last_error())


def _ptr(t):
    if t is None:
        return None
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def make_config(cfg) -> domino_config:
    """domino_config from any object with the DominoConfig fields."""
    return domino_config(
        hidden=cfg.hidden, n_layers=cfg.n_layers, n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads,
        head_dim=cfg.head_dim, ffn=cfg.ffn, vocab=cfg.vocab, block=cfg.block,
        gru_hidden=cfg.gru_hidden, rank=cfg.rank, mask_token_id=cfg.mask_id,
        rms_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
        dtype=DOMINO_BF16 if cfg.dtype == "bf16" else DOMINO_F32,
        ctx_fuse_layers=getattr(cfg, "ctx_fuse_layers", 0))


class DominoModel:
    """Owns a domino_model_t; keeps the borrowed weight tensors alive."""

    def __init__(self, cfg, dev_weights: dict, target: bool = False):
        """target=True creates a target decoder (domino_target_create): the
        Domino-head weights are not needed."""
        lib = load()
        self.cfg = cfg
        self._w = dev_weights
        L = cfg.n_layers
        self._arrays = {}

        def arr(key):
            a = (C.c_void_p * L)(*[t.data_ptr() for t in (lw[key] for lw in dev_weights["layers"])])
            self._arrays[key] = a
            return C.cast(a, _PP)

        w = domino_weights(
            embed=dev_weights["embed"].data_ptr(), lm_head=dev_weights["lm_head"].data_ptr(),
            final_norm=dev_weights["final_norm"].data_ptr(),
            attn_norm=arr("attn_norm"), wq=arr("wq"), wk=arr("wk"), wv=arr("wv"),
            q_norm=arr("q_norm"), k_norm=arr("k_norm"), wo=arr("wo"), ffn_norm=arr("ffn_norm"),
            w_gate=arr("w_gate"), w_up=arr("w_up"), w_down=arr("w_down"),
            **{k: (dev_weights[k].data_ptr() if k in dev_weights else None)
               for k in ("gru_w_ih", "gru_w_hh", "gru_b_ih", "gru_b_hh", "w1", "w2", "ctx_fc")})
        self._cfg_struct = make_config(cfg)
        h = C.c_void_p()
        create = lib.domino_target_create if target else lib.domino_model_create
        _check(create(C.byref(self._cfg_struct), C.byref(w), C.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            load().domino_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_bytes(self, batch, max_ctx, max_new, branch) -> int:
        n = load().domino_workspace_bytes(self.handle, batch, max_ctx, max_new, branch)
        if n == 0:
            raise DominoError(DOMINO_ERR_INVALID_ARG, "domino_workspace_bytes returned 0: " + last_error())
        return n


def _check_ctx_hidden(model: DominoModel, batch, ctx_hidden_new, n_new):
    """The appended rows must be fp32 and hold batch * n_new rows of the
    model's context width (k*d with k fused layers, else d)."""
    if ctx_hidden_new is None or int(n_new) <= 0:
        return
    import torch
    cfg = model.cfg
    k = getattr(cfg, "ctx_fuse_layers", 0)
    width = cfg.hidden * k if k > 0 else cfg.hidden
    need = int(batch) * int(n_new) * width
    if ctx_hidden_new.dtype != torch.float32 or not ctx_hidden_new.is_contiguous() \
            or ctx_hidden_new.numel() < need:
        raise DominoError(DOMINO_ERR_INVALID_ARG,
                          f"ctx_hidden_new must be contiguous fp32 with >= {need} elements "
                          f"([{batch}][{n_new}][{width}])")


def domino_draft_step(model: DominoModel, anchor, ctx_lens, ctx_k, ctx_v, max_ctx, topk_ids, topk_vals,
                      workspace, branch=1, ctx_hidden_new=None, n_new=0, forced=None, debug=None,
                      stream=None):
    dbg = None
    if debug:
        dbg = domino_debug(**{k: (debug[k].data_ptr() if debug.get(k) is not None else None)
                              for k in ("hidden", "base_logits", "final_logits", "states")})
    _check_ctx_hidden(model, anchor.shape[0], ctx_hidden_new, n_new)
    _check(load().domino_draft_step(
        model.handle, int(anchor.shape[0]), _ptr(anchor), _ptr(ctx_lens), _ptr(ctx_k), _ptr(ctx_v),
        int(max_ctx), _ptr(ctx_hidden_new), int(n_new), int(branch), _ptr(forced), _ptr(topk_ids),
        _ptr(topk_vals), C.byref(dbg) if dbg is not None else None, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def domino_draft_step_sampled(model: DominoModel, anchor, ctx_lens, ctx_k, ctx_v, max_ctx, topk_ids, topk_vals,
                              final_logits, workspace, temperature, seed, ctx_hidden_new=None, n_new=0,
                              forced=None, debug=None, stream=None):
    dbg = None
    if debug:
        dbg = domino_debug(**{k: (debug[k].data_ptr() if debug.get(k) is not None else None)
                              for k in ("hidden", "base_logits", "final_logits", "states")})
    _check_ctx_hidden(model, anchor.shape[0], ctx_hidden_new, n_new)
    _check(load().domino_draft_step_sampled(
        model.handle, int(anchor.shape[0]), _ptr(anchor), _ptr(ctx_lens), _ptr(ctx_k), _ptr(ctx_v),
        int(max_ctx), _ptr(ctx_hidden_new), int(n_new), float(temperature), int(seed) & (2**64 - 1),
        _ptr(forced), _ptr(topk_ids), _ptr(topk_vals), _ptr(final_logits),
        C.byref(dbg) if dbg is not None else None, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def domino_train_workspace_bytes(model: DominoModel, batch, max_ctx, max_new=0) -> int:
    n = load().domino_train_workspace_bytes(model.handle, batch, max_ctx, max_new)
    if n == 0:
        raise DominoError(DOMINO_ERR_INVALID_ARG, "domino_train_workspace_bytes returned 0: " + last_error())
    return int(n)


def domino_train_forward(model: DominoModel, anchor, ctx_lens, ctx_k, ctx_v, max_ctx, labels, lam, gamma, loss,
                         workspace, ce=None, ctx_hidden_new=None, n_new=0, debug=None, stream=None):
    dbg = None
    if debug:
        dbg = domino_debug(**{k: (debug[k].data_ptr() if debug.get(k) is not None else None)
                              for k in ("hidden", "base_logits", "final_logits", "states")})
    _check_ctx_hidden(model, anchor.shape[0], ctx_hidden_new, n_new)
    _check(load().domino_train_forward(
        model.handle, int(anchor.shape[0]), _ptr(anchor), _ptr(ctx_lens), _ptr(ctx_k), _ptr(ctx_v),
        int(max_ctx), _ptr(ctx_hidden_new), int(n_new), _ptr(labels), float(lam), float(gamma), _ptr(loss),
        _ptr(ce), C.byref(dbg) if dbg is not None else None, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def domino_target_workspace_bytes(target: DominoModel, batch, n_nodes, max_ctx) -> int:
    n = load().domino_target_workspace_bytes(target.handle, batch, n_nodes, max_ctx)
    if n == 0:
        raise DominoError(DOMINO_ERR_INVALID_ARG, "domino_target_workspace_bytes returned 0: " + last_error())
    return int(n)


def domino_target_verify(target: DominoModel, node_token, node_pos, ancestor_mask, ctx_lens, ctx_k, ctx_v, max_ctx,
                         logits, workspace, stream=None):
    import torch
    bs, nn = node_token.shape
    dt = DOMINO_BF16 if logits.dtype == torch.bfloat16 else DOMINO_F32
    _check(load().domino_target_verify(target.handle, bs, nn, _ptr(node_token), _ptr(node_pos), _ptr(ancestor_mask),
                                       _ptr(ctx_lens), _ptr(ctx_k), _ptr(ctx_v), int(max_ctx), _ptr(logits), dt,
                                       _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))


def domino_target_commit(target: DominoModel, n_nodes, ctx_lens, accept_len, accepted_nodes, ctx_k, ctx_v, max_ctx,
                         new_ctx_lens, workspace, stream=None):
    bs, max_depth = accepted_nodes.shape
    _check(load().domino_target_commit(target.handle, bs, int(n_nodes), int(max_depth), _ptr(ctx_lens),
                                       _ptr(accept_len), _ptr(accepted_nodes), _ptr(ctx_k), _ptr(ctx_v), int(max_ctx),
                                       _ptr(new_ctx_lens), _ptr(workspace), _stream(stream)))


def domino_verify_sample_workspace_bytes(batch, block, vocab) -> int:
    return int(load().domino_verify_sample_workspace_bytes(batch, block, vocab))


def domino_verify_sample(node_token, target_logits, draft_logits, temperature, seed, accept_len, accepted_nodes,
                         out_tokens, workspace, stream=None):
    import torch
    bs, B, V = target_logits.shape
    dt = DOMINO_BF16 if target_logits.dtype == torch.bfloat16 else DOMINO_F32
    _check(load().domino_verify_sample(bs, B, V, _ptr(node_token), _ptr(target_logits), dt, _ptr(draft_logits),
                                       float(temperature), int(seed) & (2**64 - 1), _ptr(accept_len),
                                       _ptr(accepted_nodes), _ptr(out_tokens), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))


def domino_philox4x32_10(counters, key, out, stream=None):
    _check(load().domino_philox4x32_10(_ptr(counters), int(key) & (2**64 - 1), _ptr(out),
                                       int(counters.shape[0]), _stream(stream)))


def domino_build_tree(topk_ids, anchor, ctx_lens, node_token, node_parent, node_depth, node_pos,
                      ancestor_mask=None, stream=None):
    bs, depth, beta = topk_ids.shape
    _check(load().domino_build_tree(bs, depth, beta, _ptr(topk_ids), _ptr(anchor), _ptr(ctx_lens),
                                    _ptr(node_token), _ptr(node_parent), _ptr(node_depth), _ptr(node_pos),
                                    _ptr(ancestor_mask), _stream(stream)))


def domino_verify_workspace_bytes(batch, n_nodes, vocab) -> int:
    return int(load().domino_verify_workspace_bytes(batch, n_nodes, vocab))


def domino_verify_accept(node_token, node_parent, target_logits, block, accept_len, accepted_nodes,
                         out_tokens, workspace, stream=None):
    import torch
    bs, nn, V = target_logits.shape
    dt = DOMINO_BF16 if target_logits.dtype == torch.bfloat16 else DOMINO_F32
    _check(load().domino_verify_accept(bs, nn, V, int(block), _ptr(node_token), _ptr(node_parent),
                                       _ptr(target_logits), dt, _ptr(accept_len), _ptr(accepted_nodes),
                                       _ptr(out_tokens), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 4 << 20


def domino_verify_accept_noalloc(node_token, node_parent, target_logits, block, accept_len, accepted_nodes,
                                 out_tokens, error_word, stream=None):
    """Greedy acceptance without a workspace (the library's fixed per-GPU scratch);
    error_word is a device int32 [1] output."""
    import torch
    bs, nn, V = target_logits.shape
    dt = DOMINO_BF16 if target_logits.dtype == torch.bfloat16 else DOMINO_F32
    _check(load().domino_verify_accept_noalloc(bs, nn, V, int(block), _ptr(node_token), _ptr(node_parent),
                                               _ptr(target_logits), dt, _ptr(accept_len), _ptr(accepted_nodes),
                                               _ptr(out_tokens), _ptr(error_word), _stream(stream)))


def domino_workspace_error(workspace, stream=None) -> int:
    v = C.c_int32(0)
    st = load().domino_workspace_error(_ptr(workspace), _stream(stream), C.byref(v))
    if st not in (DOMINO_OK, DOMINO_ERR_DEVICE):
        _check(st)
    return int(v.value)


def domino_profile_enable(model: DominoModel, classes):
    mask = 0
    for c in classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    _check(load().domino_profile_enable(model.handle, mask))


def domino_profile_reset(model: DominoModel):
    _check(load().domino_profile_reset(model.handle))


def domino_debug_set_poll_limit(model: DominoModel, polls: int):
    """Test hook: polls a persistent-rollout wait makes before it gives up (0:
    every wait gives up at once; negative: the default)."""
    _check(load().domino_debug_set_poll_limit(model.handle, int(polls)))


PATH_PERSISTENT_ROLLOUT = 1


def domino_debug_last_paths(model: DominoModel) -> int:
    """DOMINO_PATH_* bits of the execution paths the model's last draft step launched."""
    v = C.c_uint32(0)
    _check(load().domino_debug_last_paths(model.handle, C.byref(v)))
    return int(v.value)


def domino_profile_read(model: DominoModel, cls: str):
    ms, n = C.c_double(0), C.c_int32(0)
    _check(load().domino_profile_read(model.handle, KERNEL_CLASSES.index(cls), C.byref(ms), C.byref(n)))
    return float(ms.value), int(n.value)


# ---------------------------------------------------------------------------
# device marshalling helpers (torch used for memory only)
# ---------------------------------------------------------------------------
def to_device_weights(w: dict, cfg, device="cuda") -> dict:
    """Copy a numpy weight dict to device tensors in the config's storage type."""
    import torch
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def cv(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device).to(dt).contiguous()

    out = {k: cv(v) for k, v in w.items() if k != "layers"}
    out["layers"] = [{k: cv(v) for k, v in lw.items()} for lw in w["layers"]]
    return out
