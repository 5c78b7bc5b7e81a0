"""Helpers for the GPU parity tests: drive the library through the C ABI and
hand the same inputs to the oracle.

Inputs come from synth.py (weights, tokens, edits, synthetic stale caches)
or, for the small shapes, from the oracle's own prefill; no oracle input is
ever produced by the HIP path.
"""
from __future__ import annotations

import sys
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

import paper_2609_17983_amd as kvr
from oracle import decoder as od

TOL = {kvr.KVR_F32: 1e-5, kvr.KVR_BF16: 2e-2}


def say(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def relmax(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.size == 0:
        return 0.0
    return float(np.max(np.abs(a - b)) / max(float(np.max(np.abs(b))), 1e-300))


class OracleWeights:
    """Weights held as torch tensors (any device), served to the oracle as
    float64 numpy arrays one layer at a time (exact upcast)."""

    def __init__(self, w: Dict[str, object], cache: bool = False):
        self.w = w
        self._cache = {} if cache else None
        self.final_norm = w["final_norm"].to(torch.float64).cpu().numpy()

    def embed_rows(self, ids):
        idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device=self.w["embed"].device)
        return self.w["embed"][idx].to(torch.float64).cpu().numpy()

    def layer(self, l: int):
        if self._cache is not None and l in self._cache:
            return self._cache[l]
        lw = {k: (None if v is None else v.to(torch.float64).cpu().numpy()) for k, v in self.w["layers"][l].items()}
        if self._cache is not None:
            self._cache[l] = lw
        return lw


class Engine:
    """A kvr context over device weights (torch tensors)."""

    def __init__(self, shape, weights: Dict[str, object], dtype: int, max_ctx: int, max_rows: int):
        self.shape = shape
        self.dtype = dtype
        self.tdtype = torch.bfloat16 if dtype == kvr.KVR_BF16 else torch.float32
        self.weights = weights
        self.dims = kvr.dims_for(shape, dtype, max_ctx, max_rows)
        self.ws = kvr.weights_struct(weights)
        self.ctx = kvr.kvr_create(self.dims, self.ws)

    def close(self):
        if self.ctx:
            kvr.kvr_destroy(self.ctx)
            self.ctx = None

    def new_cache(self, n_cap: int) -> torch.Tensor:
        s = self.shape
        return torch.zeros((s.n_layers, 2, s.n_kv_heads, n_cap, s.head_dim), dtype=self.tdtype, device="cuda")

    def prefill(self, tokens: torch.Tensor, cache: torch.Tensor, hidden: Optional[torch.Tensor] = None,
                n: Optional[int] = None):
        n = tokens.numel() if n is None else n
        kvr.kvr_prefill(self.ctx, tokens.data_ptr(), n, cache.shape[3], cache.data_ptr(),
                        None if hidden is None else hidden.data_ptr(), torch.cuda.current_stream().cuda_stream)

    def repair(self, docs: List[dict]):
        """docs: dicts with cache, tokens, edit_start, edit_end, positions, hidden (optional), n."""
        structs = [kvr.make_doc(d["cache"].data_ptr(), d.get("n", d["tokens"].numel()), d["cache"].shape[3],
                                d["tokens"].data_ptr(), d["edit_start"], d["edit_end"], list(d["positions"]),
                                None if d.get("hidden") is None else d["hidden"].data_ptr()) for d in docs]
        kvr.kvr_repair(self.ctx, structs, torch.cuda.current_stream().cuda_stream)


def to_device_weights(w: Dict[str, object], device: str = "cuda") -> Dict[str, object]:
    return {"embed": w["embed"].to(device), "final_norm": w["final_norm"].to(device),
            "layers": [{k: (None if v is None else v.to(device)) for k, v in lw.items()} for lw in w["layers"]]}


def compare_repair(shape, stale_np: np.ndarray, stale_dev: torch.Tensor, after_dev: torch.Tensor,
                   hidden_dev: Optional[torch.Tensor], oracle_cache: np.ndarray, oracle_y: np.ndarray,
                   P: Sequence[int], n: int, tol: float, tag: str = "") -> Dict[str, float]:
    """Repaired K/V rows of P per layer and the hidden rows within `tol`
    (max |gpu - ref| / max |ref| per tensor group); every slot outside P
    bitwise unchanged."""
    P = np.asarray(P, dtype=np.int64)
    errs = {}
    after = after_dev.to(torch.float64).cpu().numpy()
    for l in range(shape.n_layers):
        for kv, name in ((0, "K"), (1, "V")):
            e = relmax(after[l, kv][:, P], oracle_cache[l, kv][:, P])
            errs[f"{name}{l}"] = e
    if hidden_dev is not None:
        errs["hidden"] = relmax(hidden_dev.cpu().numpy(), oracle_y)
    worst = max(errs, key=errs.get)
    say(f"{tag} worst {worst}={errs[worst]:.3e} (tol {tol:g})")
    assert errs[worst] <= tol, (tag, worst, errs[worst])
    mask = np.ones(stale_dev.shape[3], dtype=bool)
    mask[P] = False
    keep = torch.as_tensor(np.nonzero(mask)[0], device=stale_dev.device)
    assert torch.equal(after_dev.index_select(3, keep), stale_dev.index_select(3, keep)), f"{tag}: slots outside P changed"
    return errs
