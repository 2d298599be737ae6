"""One DP-SGD gradient step over a workload, as a sequence of C-ABI calls.

The step (section 1 and figure 1 of the paper): per-sample gradients of every
layer from its stored activations and backprops, per-sample l2 norms over all
parameters, clip factors, the clipped sum over the batch, Gaussian noise,
division by the batch size.  Every arithmetic step runs in libdpgrad's HIP
kernels; this module only owns the device buffers (allocated once, up front)
and enqueues the calls, in order, on one stream.

For a Linear layer the clipped sum is formed one of two ways, whichever moves
fewer bytes / flops at the roofline: a column reduction over the stored
per-sample gradients (reads N*P floats) or the fused GEMM B^T diag(c) A
(reads A and B again, 2*N*T*d_in*d_out flops).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional

import numpy as np

from . import binding as dp
from . import workloads as W

HBM_BYTES_PER_S = 8.0e12
# matrix-core peaks used by the clipped-sum cost model (the fused GEMM runs on
# fp32 MFMA for both input dtypes)
FUSED_FLOPS_PER_S = {W.F32: 157.3e12, W.BF16: 157.3e12}


@dataclass
class LayerBufs:
    layer: object
    A: object = None
    B: object = None
    ids: object = None
    gW: object = None
    gb: object = None
    row_ptr: object = None
    uniq: object = None
    rows: object = None
    clip_mode: str = "colreduce"


def _torch():
    import torch
    return torch


def to_device(a: np.ndarray, dtype: str, device):
    torch = _torch()
    if a.dtype == np.int64:
        return torch.from_numpy(a).to(device)
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == W.BF16:
        t = t.to(torch.bfloat16)
    return t.to(device).contiguous()


def linear_clip_mode(layer: W.Linear, N: int, dtype: str) -> str:
    elt = 2 if dtype == W.BF16 else 4
    fused = (2.0 * N * layer.T * layer.d_in * layer.d_out / FUSED_FLOPS_PER_S[dtype]
             + N * layer.T * (layer.d_in + layer.d_out) * elt / HBM_BYTES_PER_S)
    col = N * layer.n_params * 4 / HBM_BYTES_PER_S
    return "fused" if fused < col else "colreduce"


class DPStep:
    """Device buffers and the ordered calls of one DP-SGD step."""

    def __init__(self, wl: W.Workload, inputs: List[W.LayerInputs], device="cuda", C=None, sigma=None,
                 denom=None, scale=None, clip_mode: str = "auto", seed: Optional[int] = None):
        torch = _torch()
        self.wl = wl
        self.device = torch.device(device)
        self.N = int(inputs[0].B.shape[0])
        self.C = float(wl.C if C is None else C)
        self.sigma = float(wl.sigma if sigma is None else sigma)
        self.denom = float(self.N if denom is None else denom)
        self.scale = float(wl.scale if scale is None else scale)
        self.seed = int(wl.seed if seed is None else seed)
        self.dt = dp.DP_BF16 if wl.dtype == W.BF16 else dp.DP_F32
        N = self.N
        f32 = dict(dtype=torch.float32, device=self.device)
        self.layers: List[LayerBufs] = []
        ws_need = 0
        for li in inputs:
            layer = li.layer
            lb = LayerBufs(layer)
            if li.A is not None:
                lb.A = to_device(li.A, wl.dtype, self.device)
            lb.B = to_device(li.B, wl.dtype, self.device)
            if isinstance(layer, W.Linear):
                lb.gW = torch.empty((N, layer.d_out, layer.d_in), **f32)
                lb.gb = torch.empty((N, layer.d_out), **f32) if layer.bias else None
                lb.clip_mode = linear_clip_mode(layer, N, wl.dtype) if clip_mode == "auto" else clip_mode
                ws_need = max(ws_need, dp.dp_grad_sample_linear_workspace_bytes(N, layer.T, layer.d_in,
                                                                                layer.d_out, self.dt))
                if lb.clip_mode == "fused":
                    ws_need = max(ws_need, dp.dp_clip_accumulate_linear_workspace_bytes(
                        N, layer.T, layer.d_in, layer.d_out, self.dt))
                else:
                    ws_need = max(ws_need, dp.dp_clip_accumulate_workspace_bytes(N, layer.d_out * layer.d_in))
            elif isinstance(layer, W.Conv2d):
                lb.gW = torch.empty((N, layer.c_out, layer.c_in) + tuple(layer.k), **f32)
                lb.gb = torch.empty((N, layer.c_out), **f32) if layer.bias else None
                ws_need = max(ws_need, dp.dp_grad_sample_conv2d_workspace_bytes(N, layer.c_in, layer.c_out,
                                                                                *layer.k))
                ws_need = max(ws_need, dp.dp_clip_accumulate_workspace_bytes(N, layer.n_params))
            elif isinstance(layer, W.Embedding):
                lb.ids = to_device(li.ids, "", self.device)
                cap = N * layer.T
                lb.row_ptr = torch.empty(N + 1, dtype=torch.int64, device=self.device)
                lb.uniq = torch.empty(max(cap, 1), dtype=torch.int64, device=self.device)
                lb.rows = torch.empty((max(cap, 1), layer.D), **f32)
                ws_need = max(ws_need, dp.dp_grad_sample_embedding_workspace_bytes(N, layer.T))
            elif isinstance(layer, W.LayerNorm):
                lb.gW = torch.empty((N, layer.D), **f32)
                lb.gb = torch.empty((N, layer.D), **f32)
                ws_need = max(ws_need, dp.dp_grad_sample_layernorm_workspace_bytes(N, layer.T, layer.D))
                ws_need = max(ws_need, dp.dp_clip_accumulate_workspace_bytes(N, layer.D))
            self.layers.append(lb)
        self.ws = torch.empty(max(ws_need, 256), dtype=torch.uint8, device=self.device)
        self.sqnorm = torch.empty((len(self.layers), N), **f32)
        self.norm = torch.empty(N, **f32)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.params = wl.param_tensors()
        self.S: Dict[str, object] = {}
        self.out: Dict[str, object] = {}
        for name, shape in self.params:
            self.S[name] = torch.empty(shape, **f32)
            self.out[name] = torch.empty(shape, **f32)

    # ------------------------------------------------------------------ pieces
    def grad_sample(self, i: int, stream=None):
        lb = self.layers[i]
        layer = lb.layer
        N, s, sq = self.N, self.scale, self.sqnorm[i]
        if isinstance(layer, W.Linear):
            dp.dp_grad_sample_linear(lb.A, lb.B, self.dt, N, layer.T, layer.d_in, layer.d_out, s, lb.gW, lb.gb,
                                     sq, self.status, self.ws, stream)
        elif isinstance(layer, W.Conv2d):
            ho, wo = layer.out_hw
            dp.dp_grad_sample_conv2d(lb.A, lb.B, self.dt, N, layer.c_in, layer.h, layer.w, layer.c_out, ho, wo,
                                     layer.k[0], layer.k[1], layer.stride[0], layer.stride[1], layer.pad[0],
                                     layer.pad[1], 1, 1, 1, s, lb.gW, lb.gb, sq, self.status, self.ws, stream)
        elif isinstance(layer, W.Embedding):
            dp.dp_grad_sample_embedding(lb.ids, lb.B, self.dt, N, layer.T, layer.V, layer.D, s, lb.row_ptr,
                                        lb.uniq, lb.rows, N * layer.T, sq, self.status, self.ws, stream)
        elif isinstance(layer, W.LayerNorm):
            dp.dp_grad_sample_layernorm(lb.A, lb.B, self.dt, N, layer.T, layer.D, s, lb.gW, lb.gb, sq,
                                        self.status, self.ws, stream)

    def norms(self, stream=None):
        dp.dp_per_sample_norms(self.sqnorm, len(self.layers), self.N, self.norm, self.status, stream)

    def clip_sum(self, i: int, stream=None):
        lb = self.layers[i]
        layer = lb.layer
        N, C = self.N, self.C
        name = layer.name
        if isinstance(layer, W.Linear) and lb.clip_mode == "fused":
            dp.dp_clip_accumulate_linear(lb.A, lb.B, self.dt, N, layer.T, layer.d_in, layer.d_out, self.scale,
                                         self.norm, C, self.S[name + ".weight"], self.S.get(name + ".bias"),
                                         self.status, self.ws, stream)
        elif isinstance(layer, W.Embedding):
            dp.dp_clip_accumulate_embedding(lb.row_ptr, lb.uniq, lb.rows, self.norm, C, N, layer.V, layer.D,
                                            self.S[name + ".weight"], self.status, stream)
        else:
            for key, g in (("weight", lb.gW), ("bias", lb.gb)):
                if g is None:
                    continue
                numel = g[0].numel() if N > 0 else int(np.prod(self.S[name + "." + key].shape))
                dp.dp_clip_accumulate(g, self.norm, C, N, numel, self.S[name + "." + key], None,
                                      self.status, self.ws, stream)

    def noise(self, step: int, stream=None):
        for pidx, (name, shape) in enumerate(self.params):
            S = self.S[name]
            dp.dp_add_noise(S, self.out[name], S.numel(), self.seed, step, pidx, self.sigma, self.C, self.denom,
                            self.status, stream)

    # ------------------------------------------------------------------ whole step
    def run(self, step: int = 0, stream=None, mark: Optional[Callable[[str, str], None]] = None):
        """Enqueue one whole step; nothing is synchronized here."""
        self.status.zero_()
        for i, lb in enumerate(self.layers):
            if mark: mark("grad:" + lb.layer.name, "start")
            self.grad_sample(i, stream)
            if mark: mark("grad:" + lb.layer.name, "end")
        self.norms(stream)
        for i, lb in enumerate(self.layers):
            if mark: mark("clip:" + lb.layer.name, "start")
            self.clip_sum(i, stream)
            if mark: mark("clip:" + lb.layer.name, "end")
        if mark: mark("noise", "start")
        self.noise(step, stream)
        if mark: mark("noise", "end")

    def results(self) -> Dict[str, object]:
        """Copy everything back to host numpy arrays (synchronizes)."""
        torch = _torch()
        torch.cuda.synchronize(self.device)
        res = {"grads": [], "sq_layers": self.sqnorm.cpu().numpy(), "norm": self.norm.cpu().numpy(),
               "S": {k: v.cpu().numpy() for k, v in self.S.items()},
               "out": {k: v.cpu().numpy() for k, v in self.out.items()},
               "status": int(self.status.cpu().item())}
        for lb in self.layers:
            if isinstance(lb.layer, W.Embedding):
                rp = lb.row_ptr.cpu().numpy()
                nnz = int(rp[-1])
                res["grads"].append({"csr": (rp, lb.uniq[:nnz].cpu().numpy(), lb.rows[:nnz].cpu().numpy())})
            else:
                g = {"weight": lb.gW.cpu().numpy()}
                if lb.gb is not None:
                    g["bias"] = lb.gb.cpu().numpy()
                res["grads"].append(g)
        return res
