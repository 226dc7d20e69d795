"""Move drawn workloads to the GPU (tests and benchmark only).

Copies the seeded host inputs into device tensors in the layouts the library
takes (X [T, d_in]; W in the nn.Linear layout [d_out, d_in], i.e. the paper's
W transposed; ids int32) and loads adapters into a pool.  No arithmetic of
the method happens here.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from . import LayerInputs, WorkloadSpec, draw_adapter


def _torch():
    import torch
    return torch


def bits_to_device(bits: np.ndarray, device="cuda"):
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def device_to_float(t) -> np.ndarray:
    """bf16 device tensor -> float32 numpy (exact)."""
    torch = _torch()
    b = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def pack_weight(w):
    """nn.Linear-layout device weight -> the library's packed layout."""
    from paper_2510_23346_amd import pack_weight as _pack
    out = _pack(w)
    return out


class DeviceLayer:
    """Device copies of one drawn layer: ids, per-projection X, packed W and
    out."""

    def __init__(self, layer: LayerInputs, device="cuda", T: Optional[int] = None):
        torch = _torch()
        T = layer.ids.size if T is None else T
        self.T = T
        self.ids = torch.from_numpy(np.ascontiguousarray(layer.ids[:T], dtype=np.int32)).to(device)
        self.X, self.W, self.out = [], [], []
        for pi in layer.projs:
            self.X.append(bits_to_device(pi.X_bits[:T], device))
            if pi.Wq is not None:
                from paper_2510_23346_amd import pack_weight_int4
                q = torch.from_numpy(np.ascontiguousarray(pi.Wq)).to(device)
                self.W.append(pack_weight_int4(q, bits_to_device(pi.Ws_bits, device)))
            else:
                self.W.append(pack_weight(bits_to_device(np.ascontiguousarray(pi.W_bits.T), device)))
            # NaN-filled, so an output the kernels never write cannot pass a check
            self.out.append(torch.full((T, pi.spec.d_out), float("nan"), dtype=torch.bfloat16, device=device))

    def outputs(self) -> List[np.ndarray]:
        return [device_to_float(o) for o in self.out]


def make_pool(spec: WorkloadSpec, max_tokens: Optional[int] = None, max_rank: Optional[int] = None,
              device: int = 0):
    from paper_2510_23346_amd import Pool, WEIGHT_BF16, WEIGHT_INT4_G128
    mr = max(spec.ranks) if max_rank is None else max_rank
    wf = WEIGHT_INT4_G128 if spec.weight_format == "int4_g128" else WEIGHT_BF16
    return Pool(spec.projs, spec.n_slots, mr, max_tokens or spec.T, device=device, weight_formats=wf)


def load_adapters(pool, spec: WorkloadSpec, slots: Sequence[int],
                  cache: Optional[Dict[int, object]] = None):
    """Draw (or take from ``cache``) and load the adapters of ``slots``."""
    for s in slots:
        ad = cache[s] if cache is not None and s in cache else draw_adapter(spec, int(s))
        pool.load_adapter(int(s), ad.rank, ad.scale, ad.A_bits, ad.B_bits)
