"""Seeded input generators (weights, context KV, anchors, target logits).

Every tensor draws from its own stream, PCG64(SeedSequence([seed, tensor_id,
chunk])), in chunks of 2**22 elements, so values do not depend on generation
order or thread count.  Recipe (the same for every preset):

* matrices and GRU biases: N(0, 0.02), drawn in fp32, rounded to bf16
  (round-to-nearest-even) when the preset stores bf16;
* RMSNorm / q-norm / k-norm gains: 1 (or 1 + N(0, gain_std) when a test asks
  for non-trivial gains);
* context K/V caches: N(0, 1) in the storage type (K is taken to be already
  normalised and rotated, as a target's KV cache would be);
* context hidden states (tiny preset): N(0, 1);
* anchor: uniform over the vocabulary minus the MASK id;
* target logits: either N(0, 1) or Zipf(1.1)-peaked rows with a planted
  rank-1 token (see make_target_logits).

No function here computes anything the drafting method computes.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os

import numpy as np

from .configs import DominoConfig

_CHUNK = 1 << 22

# stable tensor ids
_T_EMBED, _T_LMHEAD, _T_FINAL_NORM = 0, 1, 2
_T_GRU_WIH, _T_GRU_WHH, _T_GRU_BIH, _T_GRU_BHH, _T_W1, _T_W2 = 10, 11, 12, 13, 14, 15
_T_CTX_FC = 16
_LAYER_BASE = 100
_LAYER_KEYS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
               "attn_norm", "ffn_norm", "q_norm", "k_norm")
_T_ANCHOR, _T_CTX_K, _T_CTX_V, _T_CTX_H, _T_CTX_IDS, _T_TARGET = 1000, 1001, 1002, 1003, 1004, 1005
_T_TOPK, _T_FORCED, _T_CTXLEN, _T_APPEND_H = 1006, 1007, 1008, 1009
_TARGET_LAYER_BASE = 3000


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), returned as fp32, in place."""
    assert a.dtype == np.float32
    u = a.view(np.uint32)
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    u &= np.uint32(0xFFFF0000)
    return a


def _normal(seed: int, tid: int, shape, std: float, bf16: bool) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    nchunks = (n + _CHUNK - 1) // _CHUNK

    def fill(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tid, c])))
        seg = out[lo:hi]
        g.standard_normal(out=seg, dtype=np.float32)
        if std != 1.0:
            seg *= np.float32(std)
        if bf16:
            bf16_round(seg)

    if nchunks == 1:
        fill(0)
    else:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


def _rng(seed: int, tid: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tid, sub])))


def weight_shapes(cfg: DominoConfig) -> dict:
    """Shapes of every weight tensor, row-major [out, in]."""
    d, dh, nq, nkv = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    ds, r, V, F = cfg.gru_hidden, cfg.rank, cfg.vocab, cfg.ffn
    layer = {
        "wq": (nq * dh, d), "wk": (nkv * dh, d), "wv": (nkv * dh, d), "wo": (d, nq * dh),
        "w_gate": (F, d), "w_up": (F, d), "w_down": (d, F),
        "attn_norm": (d,), "ffn_norm": (d,), "q_norm": (dh,), "k_norm": (dh,),
    }
    out = {
        "embed": (V, d), "lm_head": (V, d), "final_norm": (d,),
        "layers": [dict(layer) for _ in range(cfg.n_layers)],
        "gru_w_ih": (3 * ds, d), "gru_w_hh": (3 * ds, ds),
        "gru_b_ih": (3 * ds,), "gru_b_hh": (3 * ds,),
        "w1": (r, d + ds), "w2": (V, r),
    }
    if cfg.ctx_fuse_layers > 0:
        out["ctx_fc"] = (d, cfg.ctx_width)  # context fusion: k target layers -> d
    return out


def head_param_count(cfg: DominoConfig, with_gru_bias: bool = False) -> int:
    """Number of Domino-head parameters in the generated weights (GRU + W1 + W2)."""
    s = weight_shapes(cfg)
    keys = ["gru_w_ih", "gru_w_hh", "w1", "w2"] + (["gru_b_ih", "gru_b_hh"] if with_gru_bias else [])
    return int(sum(int(np.prod(s[k])) for k in keys))


def make_weights(cfg: DominoConfig, seed: int = 0, gain_std: float = 0.0,
                 zero_head: bool = False, zero_wo_wdown: bool = False) -> dict:
    """Random-init weights as fp32 numpy arrays (bf16-representable for bf16 presets).

    zero_head sets W2 = 0 (the head-disabled ablation); zero_wo_wdown sets the
    attention output and FFN down projections to 0 in every layer.
    """
    bf = cfg.dtype == "bf16"
    s = weight_shapes(cfg)

    def gain(tid, shape):
        if gain_std == 0.0:
            return np.ones(shape, dtype=np.float32)
        g = 1.0 + _normal(seed, tid, shape, gain_std, False)
        return bf16_round(g) if bf else g

    w = {
        "embed": _normal(seed, _T_EMBED, s["embed"], 0.02, bf),
        "lm_head": _normal(seed, _T_LMHEAD, s["lm_head"], 0.02, bf),
        "final_norm": gain(_T_FINAL_NORM, s["final_norm"]),
        "gru_w_ih": _normal(seed, _T_GRU_WIH, s["gru_w_ih"], 0.02, bf),
        "gru_w_hh": _normal(seed, _T_GRU_WHH, s["gru_w_hh"], 0.02, bf),
        "gru_b_ih": _normal(seed, _T_GRU_BIH, s["gru_b_ih"], 0.02, bf),
        "gru_b_hh": _normal(seed, _T_GRU_BHH, s["gru_b_hh"], 0.02, bf),
        "w1": _normal(seed, _T_W1, s["w1"], 0.02, bf),
        "w2": (np.zeros(s["w2"], np.float32) if zero_head
               else _normal(seed, _T_W2, s["w2"], 0.02, bf)),
        "layers": [],
    }
    if "ctx_fc" in s:
        w["ctx_fc"] = _normal(seed, _T_CTX_FC, s["ctx_fc"], 0.02, bf)
    for li, ls in enumerate(s["layers"]):
        base = _LAYER_BASE + 16 * li
        lw = {}
        for k, shape in ls.items():
            tid = base + _LAYER_KEYS.index(k)
            if k.endswith("norm"):
                lw[k] = gain(tid, shape)
            elif zero_wo_wdown and k in ("wo", "w_down"):
                lw[k] = np.zeros(shape, np.float32)
            else:
                lw[k] = _normal(seed, tid, shape, 0.02, bf)
        w["layers"].append(lw)
    return w


def make_target_weights(cfg: DominoConfig, seed: int = 0, gain_std: float = 0.0,
                        zero_wo_wdown: bool = False) -> dict:
    """Random-init weights of a target decoder (the same recipe as the drafter's
    layers).  The embedding, LM head and final norm use the drafter's tensor ids,
    so a drafter and a target of the same width and vocabulary share them (the
    drafter reuses the target's frozen embedding and LM head); the layers have
    their own streams."""
    bf = cfg.dtype == "bf16"
    s = weight_shapes(cfg)

    def gain(tid, shape):
        if gain_std == 0.0:
            return np.ones(shape, dtype=np.float32)
        g = 1.0 + _normal(seed, tid, shape, gain_std, False)
        return bf16_round(g) if bf else g

    w = {"embed": _normal(seed, _T_EMBED, s["embed"], 0.02, bf),
         "lm_head": _normal(seed, _T_LMHEAD, s["lm_head"], 0.02, bf),
         "final_norm": gain(_T_FINAL_NORM, s["final_norm"]),
         "layers": []}
    for li, ls in enumerate(s["layers"]):
        base = _TARGET_LAYER_BASE + 16 * li
        lw = {}
        for k, shape in ls.items():
            tid = base + _LAYER_KEYS.index(k)
            if k.endswith("norm"):
                lw[k] = gain(tid, shape)
            elif zero_wo_wdown and k in ("wo", "w_down"):
                lw[k] = np.zeros(shape, np.float32)
            else:
                lw[k] = _normal(seed, tid, shape, 0.02, bf)
        w["layers"].append(lw)
    return w


def make_inputs(cfg: DominoConfig, seed: int = 0, ctx_lens=None, max_ctx: int | None = None) -> dict:
    """Anchor ids, context lengths and the context (KV cache or hidden states).

    Returns a dict with
      anchor   int32 [bs]
      ctx_lens int32 [bs]
      ctx_k, ctx_v  fp32 [L, bs, max_ctx, n_kv, d_h] (zeros when ctx_from_hidden)
      ctx_hidden    fp32 [bs, n_new, cfg.ctx_width] or None, n_new = min(ctx_lens)
    """
    bs, V = cfg.batch, cfg.vocab
    mask = cfg.mask_id
    a = _rng(seed, _T_ANCHOR).integers(0, V - 1, size=bs, dtype=np.int64)
    a = np.where(a >= mask, a + 1, a).astype(np.int32)
    if ctx_lens is None:
        ctx_lens = np.full(bs, cfg.ctx, dtype=np.int32)
    ctx_lens = np.asarray(ctx_lens, dtype=np.int32)
    mc = int(max_ctx if max_ctx is not None else max(cfg.ctx, int(ctx_lens.max(initial=0))))
    shape = (cfg.n_layers, bs, mc, cfg.n_kv_heads, cfg.head_dim)
    bf = cfg.dtype == "bf16"
    out = {"anchor": a, "ctx_lens": ctx_lens, "max_ctx": mc}
    if cfg.ctx_from_hidden:
        out["ctx_k"] = np.zeros(shape, np.float32)
        out["ctx_v"] = np.zeros(shape, np.float32)
        n_new = int(ctx_lens.min()) if ctx_lens.size else 0
        out["ctx_hidden"] = _normal(seed, _T_CTX_H, (bs, n_new, cfg.ctx_width), 1.0, bf)
        out["ctx_ids"] = _rng(seed, _T_CTX_IDS).integers(0, V - 1, size=(bs, n_new)).astype(np.int32)
    else:
        out["ctx_k"] = _normal(seed, _T_CTX_K, shape, 1.0, bf)
        out["ctx_v"] = _normal(seed, _T_CTX_V, shape, 1.0, bf)
        out["ctx_hidden"] = None
    return out


def make_append_hidden(cfg: DominoConfig, n_new: int, seed: int = 0) -> np.ndarray:
    """Target hidden states of the tokens accepted last cycle, [bs, n_new, cfg.ctx_width]
    N(0, 1) (storage-type values), to be appended to a KV-cache context."""
    return _normal(seed, _T_APPEND_H, (cfg.batch, n_new, cfg.ctx_width), 1.0, cfg.dtype == "bf16")


def make_forced_tokens(cfg: DominoConfig, seed: int = 0) -> np.ndarray:
    """Uniform draft tokens [bs, B-1] for teacher-forced runs."""
    return _rng(seed, _T_FORCED).integers(0, cfg.vocab, size=(cfg.batch, cfg.depth)).astype(np.int32)


def make_random_topk(cfg: DominoConfig, seed: int = 0, vocab: int | None = None) -> np.ndarray:
    """Distinct random token ids per position, [bs, B-1, beta] int32."""
    V = cfg.vocab if vocab is None else vocab
    g = _rng(seed, _T_TOPK)
    out = np.empty((cfg.batch, cfg.depth, cfg.branch), np.int32)
    for b in range(cfg.batch):
        for j in range(cfg.depth):
            out[b, j] = g.choice(V, size=cfg.branch, replace=False)
    return out


def _zipf_trunc(g: np.random.Generator, kmax: int, s: float = 1.1) -> int:
    p = np.arange(1, kmax + 1, dtype=np.float64) ** (-s)
    return int(g.choice(kmax, p=p / p.sum())) + 1


def make_target_logits(cfg: DominoConfig, node_token: np.ndarray, node_parent: np.ndarray,
                       seed: int = 0, kind: str = "zipf", dtype: str = "bf16",
                       vocab: int | None = None) -> np.ndarray:
    """Synthetic target logits [bs, N+1, V] as fp32 values (bf16-representable if dtype=bf16).

    kind="normal": i.i.d. N(0, 1).
    kind="zipf":   row m holds -1.1 * ln(rank) over a random permutation of the
      ranks 1..V (so its softmax is exactly Zipf(1.1)).  The rank-1 token is
      planted: draw c from Zipf(1.1) truncated to {1..beta+1}; if node m has a
      c-th child (children in node order) that child's token gets rank 1,
      otherwise a random token that is none of m's children does.
    """
    V = cfg.vocab if vocab is None else vocab
    node_token = np.asarray(node_token)
    node_parent = np.asarray(node_parent)
    bs, nn = node_token.shape
    out = np.empty((bs, nn, V), np.float32)
    if kind == "normal":
        out[...] = _normal(seed, _T_TARGET, (bs, nn, V), 1.0, dtype == "bf16")
        return out
    assert kind == "zipf"
    base = (-1.1 * np.log(np.arange(1, V + 1, dtype=np.float64))).astype(np.float32)
    if dtype == "bf16":
        bf16_round(base)

    def row(bm):
        b, m = divmod(bm, nn)
        g = _rng(seed, _T_TARGET, bm)
        perm = g.permutation(V)            # perm[v] = rank-1 of token v
        kids = [int(node_token[b, c]) for c in range(nn) if int(node_parent[b, c]) == m]
        c = _zipf_trunc(g, cfg.branch + 1)
        if c <= len(kids):
            top = kids[c - 1]
        else:
            while True:
                top = int(g.integers(0, V))
                if top not in kids:
                    break
        cur = int(np.flatnonzero(perm == 0)[0])
        perm[cur], perm[top] = perm[top], perm[cur]
        out[b, m] = base[perm]

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(row, range(bs * nn)))
    return out
