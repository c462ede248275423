"""Shared helpers for the GPU parity tests: run the HIP path through the C-ABI
binding and compare with the CPU oracle."""
import sys
import time

import numpy as np

import oracle
import synth

NEAR_TIE = 1e-3  # top-1 (and top-beta order) must agree where the oracle's gap is at least this


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


class GpuRun:
    """Model + buffers for one config on cuda:0."""

    def __init__(self, cfg, w, max_ctx, beta, n_new=0, device="cuda:0"):
        import torch
        from paper_2605_29707_amd import binding as bd
        self.torch, self.bd = torch, bd
        self.cfg, self.beta, self.max_ctx, self.n_new = cfg, beta, max_ctx, n_new
        self.dev = torch.device(device)
        self.dw = bd.to_device_weights(w, cfg, self.dev)
        self.model = bd.DominoModel(cfg, self.dw)
        bs, D, V = cfg.batch, cfg.depth, cfg.vocab
        nb = self.model.workspace_bytes(bs, max_ctx, n_new, beta)
        self.ws = torch.empty(nb, dtype=torch.uint8, device=self.dev)
        self.ids = torch.empty(bs, D, beta, dtype=torch.int32, device=self.dev)
        self.vals = torch.empty(bs, D, beta, dtype=torch.float32, device=self.dev)

    def t(self, a, dt=None):
        torch = self.torch
        dt = dt or torch.float32
        return torch.from_numpy(np.ascontiguousarray(a)).to(self.dev).to(dt)

    def kv_dtype(self):
        return self.torch.bfloat16 if self.cfg.dtype == "bf16" else self.torch.float32

    def step(self, inp, forced=None, debug=True, ctx_lens=None):
        torch, bd, cfg = self.torch, self.bd, self.cfg
        bs, D, V = cfg.batch, cfg.depth, cfg.vocab
        anchor = self.t(inp["anchor"], torch.int32)
        lens = self.t(inp["ctx_lens"] if ctx_lens is None else ctx_lens, torch.int32)
        ck = self.t(inp["ctx_k"], self.kv_dtype())
        cv = self.t(inp["ctx_v"], self.kv_dtype())
        hid = None
        if self.n_new > 0:
            hid = self.t(inp["ctx_hidden"])
        dbg = None
        if debug:
            dbg = {"hidden": torch.empty(bs, D, cfg.hidden, device=self.dev),
                   "base_logits": torch.empty(bs, D, V, device=self.dev),
                   "final_logits": torch.empty(bs, D, V, device=self.dev),
                   "states": torch.empty(bs, D, cfg.gru_hidden, device=self.dev)}
        fz = None if forced is None else self.t(forced, torch.int32)
        bd.domino_draft_step(self.model, anchor, lens, ck, cv, self.max_ctx, self.ids, self.vals, self.ws,
                             branch=self.beta, ctx_hidden_new=hid, n_new=self.n_new, forced=fz, debug=dbg)
        torch.cuda.synchronize()
        out = {"topk_ids": self.ids.cpu().numpy().copy(), "topk_vals": self.vals.cpu().numpy().copy(),
               "err": bd.domino_workspace_error(self.ws)}
        if debug:
            out.update({k: v.cpu().numpy() for k, v in dbg.items()})
        out["ctx_k"] = ck.float().cpu().numpy()
        out["ctx_v"] = cv.float().cpu().numpy()
        return out

    def close(self):
        self.model.close()


def check_against_oracle(cfg, gpu, ref, tol, beta):
    """Logit / state tolerance plus top-1 (and top-beta order) agreement away from near-ties."""
    errs = {}
    for k in ("hidden", "base_logits", "final_logits", "states"):
        errs[k] = float(np.abs(gpu[k] - ref[k]).max())
    log("max |gpu - oracle|: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v < tol, f"{k}: {v} >= {tol}"
    bs, D = gpu["topk_ids"].shape[:2]
    np.testing.assert_allclose(gpu["topk_vals"], np.take_along_axis(
        ref["final_logits"], gpu["topk_ids"].astype(np.int64), axis=2), atol=tol, rtol=0)
    checked = 0
    for b in range(bs):
        for j in range(D):
            row = ref["final_logits"][b, j]
            ids, vals = oracle.top_beta(row, beta + 1)
            gaps = -np.diff(vals)
            for q in range(beta):
                if np.all(gaps[: q + 1] >= NEAR_TIE):
                    assert gpu["topk_ids"][b, j, q] == ids[q], (b, j, q)
                    checked += 1
    return checked
