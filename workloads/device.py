"""Copy a generated workload to the GPU as the binding's argument tensors (data movement only)."""
from __future__ import annotations

import numpy as np
import torch


def to_device(w, device="cuda", row_offset_bytes: int = 0):
    """Return (logits [B, ld] tensor, uniforms, SamplingParams) on ``device``.

    ``row_offset_bytes`` (a multiple of the element size) shifts the whole matrix inside a larger
    allocation so the rows start at addresses that are not 16-byte aligned.
    """
    from paper_2606_01927_amd import SamplingParams

    if w.dtype == "bf16":
        host = torch.from_numpy(np.ascontiguousarray(w.logits).view(np.int16)).view(torch.bfloat16)
    else:
        host = torch.from_numpy(np.ascontiguousarray(w.logits, dtype=np.float32))
    if row_offset_bytes:
        es = host.element_size()
        assert row_offset_bytes % es == 0
        k = row_offset_bytes // es
        flat = torch.empty(host.numel() + k, dtype=host.dtype, device=device)
        flat[k:] = host.reshape(-1).to(device)
        logits = flat[k:].view(w.B, w.ld)
    else:
        logits = host.to(device)

    def t(a, dt):
        return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt)

    p = SamplingParams(
        temperature=t(w.temperature, torch.float32), top_k=t(w.top_k, torch.int32),
        top_p=t(w.top_p, torch.float32), min_p=t(w.min_p, torch.float32),
        repetition_penalty=t(w.repetition_penalty, torch.float32),
        frequency_penalty=t(w.frequency_penalty, torch.float32),
        presence_penalty=t(w.presence_penalty, torch.float32),
        hist_offsets=t(w.hist_offsets, torch.int64), hist_ids=t(w.hist_ids, torch.int32),
        prompt_offsets=t(getattr(w, "prompt_offsets", None), torch.int64),
        prompt_ids=t(getattr(w, "prompt_ids", None), torch.int32))
    u = t(w.uniforms, torch.float32)
    return logits, u, p
