"""CPU oracle for temperature sampling in drafting and verification.

TEST INFRASTRUCTURE ONLY (same rules as domino_oracle: only the tests, the
package smoke check and the benchmark's CPU-baseline leg use it; it shares no
code with the GPU path).  Float64 throughout.

What it follows:

* Fig. 3 caption / Sec. 4.1.2: at temperature T each draft token is sampled
  from the final logits l_i + c_i, i.e. from softmax((l_i + c_i) / T), and fed
  back into the causal state.
* Sec. 3.1: the target accepts the longest valid prefix "according to the
  standard speculative verification rule" (the rejection-sampling rule of the
  speculative-sampling papers it cites): draft token x at depth j, drawn from
  q_j, is accepted with probability min(1, p_j(x) / q_j(x)); at the first
  rejection the bonus token is drawn from the residual max(0, p_j - q_j)
  (normalised); if every draft token is accepted the bonus is drawn from the
  target's next distribution p_{B}.  tau = accepted + 1.
* Readings (the paper gives no sampler): every random draw comes from the
  counter-based generator Philox-4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
  random numbers: as easy as 1, 2, 3", SC 2011) keyed by the 64-bit seed, so a
  draw is a pure function of (seed, stream, batch row, depth, vocabulary id):
    counter = (v // 4, depth, row, stream), key = (seed lo, seed hi),
    word v % 4 of the output; stream 0 = draft noise, 1 = acceptance uniform
    (v = 0), 2 = bonus noise.
  A word x becomes the uniform u = (floor(x / 2^9) + 1/2) / 2^23 in (0, 1),
  which is exactly representable in fp32 (so a GPU forms the same value).
  Sampling from softmax(z) is the Gumbel-max form argmax_v (z_v + g_v) with
  g_v = -log(-log u_v) (exactly a draw from softmax(z)); ties by lower id,
  NaN as -inf.  Sampling from a normalised nonnegative vector w is the same
  with z_v = log w_v over w_v > 0.  Only the chain (one token per depth) is
  verified this way.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64
M0, M1 = 0xD2511F53, 0xCD9E8D57      # Philox-4x32 multipliers (Salmon et al. 2011)
W0, W1 = 0x9E3779B9, 0xBB67AE85      # Weyl key increments
STREAM_DRAFT, STREAM_ACCEPT, STREAM_BONUS = 0, 1, 2
MASK32 = 0xFFFFFFFF


def philox4x32_10(counter, key):
    """Philox-4x32 with 10 rounds.

    counter: uint32 array [..., 4]; key: two uint32 words.  Each round maps
    (c0, c1, c2, c3) to (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
    lo(M0 c0)); the key advances by (W0, W1) between rounds.
    """
    c = np.asarray(counter, dtype=np.uint64) & MASK32
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for r in range(10):
        if r > 0:
            k0, k1 = (k0 + W0) & MASK32, (k1 + W1) & MASK32
        p0 = np.uint64(M0) * c0
        p1 = np.uint64(M1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(MASK32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(MASK32)
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def seed_key(seed):
    return (int(seed) & MASK32, (int(seed) >> 32) & MASK32)


def uniform01(x):
    """Word -> uniform in (0, 1): (floor(x / 2^9) + 1/2) / 2^23."""
    x = np.asarray(x, dtype=np.uint64)
    return ((x >> np.uint64(9)).astype(F64) + 0.5) / F64(1 << 23)


def words(seed, stream, row, depth, n):
    """Words v = 0..n-1 of (seed, stream, row, depth)."""
    v = np.arange(n, dtype=np.int64)
    ctr = np.stack([v // 4, np.full(n, depth), np.full(n, row), np.full(n, stream)], axis=-1)
    out = philox4x32_10(ctr, seed_key(seed))
    return out[np.arange(n), v % 4]


def gumbel(u):
    return -np.log(-np.log(np.asarray(u, F64)))


def gumbel_argmax(z, g):
    """argmax_v (z_v + g_v) under (value desc, id asc), NaN as -inf.

    Returns (token, gap between the best and second-best keys)."""
    key = np.asarray(z, F64) + np.asarray(g, F64)
    key[np.isnan(key)] = -np.inf
    m = np.max(key)
    tok = int(np.flatnonzero(key == m)[0])
    rest = np.delete(key, tok)
    gap = float(m - np.max(rest)) if rest.size else np.inf
    return tok, gap


def sample_draft(final_row, temperature, seed, row, depth):
    """Draft token at `depth` (1-based) of batch row `row`: a draw from
    softmax(final_row / T).  Returns (token, key gap)."""
    V = np.asarray(final_row).shape[0]
    g = gumbel(uniform01(words(seed, STREAM_DRAFT, row, depth, V)))
    return gumbel_argmax(np.asarray(final_row, F64) / F64(temperature), g)


def softmax_t(logits, temperature):
    z = np.asarray(logits, F64) / F64(temperature)
    z = z - np.max(z)
    e = np.exp(z)
    return e / np.sum(e)


def verify_sample(node_token, target_logits, draft_logits, temperature, seed, rows=None, block=16):
    """Speculative-sampling verification of a chain of B-1 draft tokens.

    node_token: [bs, B] (node 0 = the anchor, node j = the draft token at depth
    j); target_logits: [bs, B, V], row m = the target's distribution after node
    m; draft_logits: [bs, B-1, V], the drafter's final logits at depths 1..B-1.
    `rows` gives the batch-row index each row's random streams use (default
    0..bs-1).  Returns accept_len [bs] (tau - 1), accepted_nodes [bs, B-1] and
    out_tokens [bs, B] as the greedy rule does, plus per-row decision margins
    (|u - p/q| of each decision taken, and the bonus draw's key gap).
    """
    node_token = np.asarray(node_token)
    bs = node_token.shape[0]
    depth = block - 1
    rows = np.arange(bs) if rows is None else np.asarray(rows)
    acc_len = np.zeros(bs, np.int32)
    acc_nodes = np.full((bs, depth), -1, np.int32)
    out_tok = np.full((bs, block), -1, np.int32)
    margins, bonus_gap = [], np.zeros(bs)
    for b in range(bs):
        rb = int(rows[b])
        mrow = []
        a = 0
        stop = depth + 1  # depth whose distribution the bonus comes from
        for j in range(1, depth + 1):
            p = softmax_t(target_logits[b, j - 1], temperature)
            q = softmax_t(draft_logits[b, j - 1], temperature)
            x = int(node_token[b, j])
            u = uniform01(words(seed, STREAM_ACCEPT, rb, j, 1))[0]
            ratio = p[x] / q[x]
            mrow.append(abs(u - ratio))
            if u < ratio:                     # accepted with probability min(1, p/q)
                acc_nodes[b, a] = j
                out_tok[b, a] = x
                a += 1
                continue
            stop = j
            break
        if stop <= depth:
            p = softmax_t(target_logits[b, stop - 1], temperature)
            q = softmax_t(draft_logits[b, stop - 1], temperature)
            w = np.maximum(p - q, 0.0)
        else:
            w = softmax_t(target_logits[b, depth], temperature)
        with np.errstate(divide="ignore"):
            z = np.where(w > 0, np.log(w), -np.inf)
        g = gumbel(uniform01(words(seed, STREAM_BONUS, rb, stop, w.shape[0])))
        tok, gap = gumbel_argmax(z, g)
        acc_len[b] = a
        out_tok[b, a] = tok
        margins.append(mrow)
        bonus_gap[b] = gap
    return {"accept_len": acc_len, "accepted_nodes": acc_nodes, "out_tokens": out_tok,
            "accept_margins": margins, "bonus_gap": bonus_gap}
