"""Device-resident inputs for a synthetic layout (torch; no method arithmetic).

Full-size batches are drawn on the device with torch's generator (same
distributions as `make_values`); the rows of the users listed in `exact_users`
are then overwritten with their per-user numpy draws, so a CPU reference can
check exactly those users.  Users are independent, so the other users' values
do not influence the checked rows.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional

import numpy as np
import torch

from .batches import TOKEN_TENSORS, Layout, make_values

_QKVU = ("q", "k", "v", "u")


def device_inputs(layout: Layout, device="cuda", exact_users: Optional[Iterable[int]] = None,
                  all_exact: bool = False, tensors=TOKEN_TENSORS, torch_seed: int = 1234) -> dict:
    spec = layout.spec
    H, dh = spec.heads, spec.head_dim
    d = H * dh
    T = layout.total_tokens
    dtype = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    out = {"dtype": dtype}
    if all_exact:
        vals = make_values(layout, tensors=tensors)
        for name in tensors:
            out[name] = torch.from_numpy(vals[name]).to(device=device, dtype=dtype)
    else:
        g = torch.Generator(device=device)
        g.manual_seed(torch_seed + 7919 * layout.extra.get("seed", spec.seed))
        for name in tensors:
            shape = (T, H, dh) if name in ("q", "k", "v", "do") else (T, d)
            x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
            if name in _QKVU:
                x.mul_(1.0 / math.sqrt(dh))
            out[name] = x.to(dtype)
        exact_users = list(exact_users or [])
        if exact_users:
            vals = make_values(layout, users=exact_users, tensors=tensors)
            row = 0
            for b in exact_users:
                sl = layout.user_slice(b)
                n = sl.stop - sl.start
                for name in tensors:
                    out[name][sl] = torch.from_numpy(vals[name][row:row + n]).to(device=device, dtype=dtype)
                row += n
    params = make_values(layout, users=[], tensors=())
    out["gamma"] = torch.from_numpy(params["gamma"]).to(device)
    out["beta"] = torch.from_numpy(params["beta"]).to(device)
    out["rab"] = None if params["rab"] is None else torch.from_numpy(params["rab"]).to(device)
    out["gamma_np"], out["beta_np"], out["rab_np"] = params["gamma"], params["beta"], params["rab"]
    out["offsets"] = torch.from_numpy(layout.offsets.astype(np.int32)).to(device)
    out["seg"] = torch.from_numpy(layout.seg).to(device)
    out["ts"] = torch.from_numpy(layout.ts).to(device)
    out["max_seqlen"] = layout.max_seqlen
    return out
