"""Helpers for the GPU parity tests: device copies of generated inputs."""
import numpy as np
import torch

import paper_2502_01637_amd as S
from workloads import fill_table, torch_dtype


def dev(a, device="cuda"):
    a = np.ascontiguousarray(a)
    # a reversed axis of length 1 keeps its negative stride through
    # ascontiguousarray (the array still counts as contiguous); torch refuses it
    if any(s < 0 for s in a.strides):
        a = a.copy()
    return torch.from_numpy(a).to(device)


def build_gpu(fgrams, lengths, ids, max_load=0.5):
    return S.build_fgram_table(dev(np.asarray(fgrams, dtype=np.int32)),
                               dev(np.asarray(lengths, dtype=np.int32)),
                               dev(np.asarray(ids, dtype=np.int32)), max_load=max_load)


def device_rows(cfg, device="cuda"):
    t = torch.empty((cfg.n_rows, cfg.d), dtype=torch_dtype(cfg), device=device)
    return fill_table(cfg, t)


def as_bytes(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.uint8).cpu().numpy()
