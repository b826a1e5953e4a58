"""Helpers shared by the GPU parity tests (not collected by pytest)."""
import numpy as np
import torch

from paper_2401_04829_amd import _lib as L
from paper_2401_04829_amd.explainer import Explainer, _vp


def require_gpu():
    assert torch.cuda.is_available(), "the gpu tests need a GPU"
    L.load()                       # raises if libgnnshap.so is not built
    return torch.device("cuda:0")


def masks_np(t):
    return t.cpu().numpy().view(np.uint64)


def sample_on_gpu(M, p, seed, stream_id, device="cuda:0"):
    plan, classes = L.gnnshap_plan_samples(M, p, seed, stream_id)
    k, wpr = plan.num_rows, plan.words_per_row
    masks = torch.empty((k, wpr), dtype=torch.int64, device=device)
    weights = torch.empty(k, dtype=torch.float32, device=device)
    ws = torch.empty(max(L.gnnshap_sample_workspace(plan), 256), dtype=torch.uint8, device=device)
    s = torch.cuda.current_stream().cuda_stream
    L.gnnshap_sample_coalitions(plan, classes, _vp(masks), _vp(weights), _vp(ws), ws.numel(), s)
    torch.cuda.synchronize()
    return plan, classes, masks, weights


def y_tolerance(y_ref, f_empty, f_full):
    """|y_gpu - y_ref| <= 1e-4 * max(|y_ref|, s_v), s_v = max(|f(E_c)|, |f(empty)|)."""
    s_v = max(abs(f_empty), abs(f_full))
    return 1e-4 * np.maximum(np.abs(y_ref), s_v)


def explainer_for(cfg):
    return Explainer(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"], cfg["hops"])
