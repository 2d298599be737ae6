"""One DP-SGD gradient step over a workload, as a sequence of C-ABI calls.

The step (section 1 and figure 1 of the paper): per-sample gradients of every
layer from its stored activations and backprops, per-sample l2 norms over all
parameters, clip factors, the clipped sum over the batch, Gaussian noise,
division by the batch size.  Every arithmetic step runs in libdpgrad's HIP
kernels; this module only owns the device buffers (allocated once, up front)
and enqueues the calls, in order, on one stream:

  1. one per-sample-gradient call per layer (each also writes that layer's
     row of per-sample squared norms);
  2. dp_per_sample_norms, when a fused clipped sum needs the norms first;
  3. fused clipped sums where they are cheaper (Linear: B^T diag(c) A, all
     layers in one grouped call; Embedding: CSR -> dense);
  4. one dp_norms_clip_noise launch for every parameter tensor: the norms
     (unless step 2 ran), the column reductions of the remaining per-sample
     gradients, and every tensor's noised average.

A step can be captured once as a HIP graph and replayed; the noise step then
comes from a device counter that the graph advances itself.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import binding as dp
from . import workloads as W

# Effective rates measured on MI355X for the clipped-sum route choice (not
# spec peaks): the column reduction streams at ~4.5 TB/s; the fused GEMM
# reaches ~60 TFLOP/s on fp32 MFMA, ~190 TFLOP/s on the single-layer bf16
# path and ~650 TFLOP/s in the grouped bf16 launch (T a multiple of 32,
# feature sizes multiples of 8); each extra launch of the fused route costs
# ~3 us next to the grouped column reduction, which all tensors share.
HBM_BYTES_PER_S = 4.5e12
FUSED_FLOPS_PER_S = {W.F32: 60e12, W.BF16: 60e12}
BF16_FLOPS_PER_S = 190e12
BF16_GROUPED_FLOPS_PER_S = 650e12
LAUNCH_S = 3e-6


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
    ghost: bool = False         # norm from the Gram matrices, no per-sample gradient
    ws: object = None          # scratch of the per-sample-gradient call
    ws_clip: object = None     # scratch of the fused clipped sum
    aux: object = None         # LSTMRecurrence: stored gates, cell states, W_hh, dh_last


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
    """'fused' (B^T diag(c) A from A and B) or 'colreduce' (read the stored grads)."""
    elt = 2 if dtype == W.BF16 else 4
    bf16_mfma = dtype == W.BF16 and layer.T > 1 and layer.d_in % 8 == 0 and layer.d_out % 8 == 0
    grouped = bf16_mfma and layer.T % 32 == 0
    peak = BF16_GROUPED_FLOPS_PER_S if grouped else BF16_FLOPS_PER_S if bf16_mfma else FUSED_FLOPS_PER_S[dtype]
    fused = (2.0 * N * layer.T * layer.d_in * layer.d_out / peak
             + N * layer.T * (layer.d_in + layer.d_out) * elt / HBM_BYTES_PER_S + 2 * LAUNCH_S)
    col = N * layer.n_params * 4 / HBM_BYTES_PER_S
    return "fused" if fused < col else "colreduce"


class DPStep:
    """Device buffers and the ordered calls of one DP-SGD step."""

    def __init__(self, wl: W.Workload, inputs: List[W.LayerInputs], device="cuda", C=None, sigma=None,
                 denom=None, scale=None, clip_mode: str = "auto", seed: Optional[int] = None,
                 norm_mode: str = "materialize", virtual_batches: int = 1,
                 sigma_schedule: Optional[Sequence[float]] = None, variable_batch: bool = False):
        """norm_mode: 'materialize' computes every layer's per-sample gradients
        (the paper's method); 'ghost' gives a Linear layer whose clipped sum is
        fused, and for which 2 T^2 < d_in * d_out, its per-sample norm from
        the T x T Gram matrices instead, and never forms its per-sample
        gradient (weight and bias sums then both come from the fused GEMM).

        virtual_batches: K physical batches (of this step's N samples) per
        logical batch; each physical batch's clipped sums are added into a
        running sum, and only the last adds noise and divides (by K*N unless
        denom is given).  Drive it with run(reset=..., emit=...) or
        run_virtual.

        sigma_schedule: the noise multiplier per step (a noise scheduler:
        exponential, step or any custom schedule, evaluated beforehand);
        step t uses sigma_schedule[min(t, len - 1)], read on the device, so
        captured graphs follow it from replay to replay.  It replaces sigma.
        denom: the divisor of the noisy sum, e.g. the expected batch size
        q * dataset size under Poisson sampling (the default is the physical
        batch times virtual_batches).

        variable_batch: the step's N rows hold a batch of variable size (the
        Poisson-sampled batch, padded to N rows); set_active(n) sets its size
        in device memory, so a captured graph follows it from replay to
        replay.  Rows past it still have their per-sample gradients formed
        (fixed shapes) but get the norm -1 and clip factor 0, and add nothing
        to the sums; they must hold finite values.  Pass denom (the expected
        batch size) with it."""
        torch = _torch()
        self.wl = wl
        self.device = torch.device(device)
        self.N = int(next(li.B.shape[0] for li in inputs if li.B is not None))
        self.C = float(wl.C if C is None else C)
        self.sigma = float(wl.sigma if sigma is None else sigma)
        self.sigma_tab = None
        if sigma_schedule is not None:
            sched = [float(x) for x in sigma_schedule]
            if not sched:
                raise ValueError("sigma_schedule needs at least one entry")
            self.sigma_tab = torch.tensor(sched, dtype=torch.float32, device=torch.device(device))
        self.n_active = None
        if variable_batch:
            if self.sigma_tab is None:   # the schedule entry point carries the batch size
                self.sigma_tab = torch.tensor([self.sigma], dtype=torch.float32, device=torch.device(device))
            self.n_active = torch.tensor([self.N], dtype=torch.int64, device=torch.device(device))
        self.virtual_batches = int(virtual_batches)
        if self.virtual_batches < 1:
            raise ValueError("virtual_batches must be >= 1")
        self.denom = float(self.N * self.virtual_batches if denom is None else denom)
        self.scale = float(wl.scale if scale is None else scale)
        self.seed = int(wl.seed if seed is None else seed)
        self.dt = dp.DP_BF16 if wl.dtype == W.BF16 else dp.DP_F32
        N = self.N
        f32 = dict(dtype=torch.float32, device=self.device)
        self.layers: List[LayerBufs] = []
        self.recurrences: Dict[str, object] = {}      # LSTMRecurrence name -> its gate backprop buffer
        for li in inputs:
            layer = li.layer
            lb = LayerBufs(layer)
            if li.A is not None:
                lb.A = to_device(li.A, wl.dtype, self.device)
            if isinstance(layer, W.LSTMRecurrence):
                # stored forward activations in, the gate backprop (B of the
                # LSTM's weight layers) out
                lb.aux = {k: to_device(v, W.F32, self.device) for k, v in li.aux.items()}
                lb.B = torch.empty((N, layer.T, 4 * layer.H), **f32)
                self.recurrences[layer.name] = lb.B
            elif getattr(layer, "bsource", None):
                lb.B = self.recurrences[layer.bsource]
            else:
                lb.B = to_device(li.B, wl.dtype, self.device)
            need_g = need_c = 0
            if isinstance(layer, W.Linear):
                lb.clip_mode = linear_clip_mode(layer, N, wl.dtype) if clip_mode == "auto" else clip_mode
                lb.ghost = (norm_mode == "ghost" and lb.clip_mode == "fused"
                            and 2 * layer.T * layer.T < layer.d_in * layer.d_out)
                if not lb.ghost:            # ghost layers share one grouped call and its workspace
                    lb.gW = torch.empty((N, layer.d_out, layer.d_in), **f32)
                    lb.gb = torch.empty((N, layer.d_out), **f32) if layer.bias else None
                    need_g = dp.dp_grad_sample_linear_workspace_bytes(N, layer.T, layer.d_in, layer.d_out, self.dt)
            elif isinstance(layer, W.Conv2d):
                lb.gW = torch.empty((N, layer.c_out, layer.c_in) + tuple(layer.k), **f32)
                lb.gb = torch.empty((N, layer.c_out), **f32) if layer.bias else None
                need_g = dp.dp_grad_sample_conv2d_workspace_bytes(
                    N, layer.c_in, layer.h, layer.w, layer.c_out, layer.k[0], layer.k[1], layer.stride[0],
                    layer.stride[1], layer.pad[0], layer.pad[1])
            elif isinstance(layer, W.Embedding):
                lb.ids = to_device(li.ids, "", self.device)
                cap = N * layer.T
                lb.row_ptr = torch.empty(N + 1, dtype=torch.int64, device=self.device)
                lb.uniq = torch.empty(max(cap, 1), dtype=torch.int64, device=self.device)
                lb.rows = torch.empty((max(cap, 1), layer.D), **f32)
                need_g = dp.dp_grad_sample_embedding_workspace_bytes(N, layer.T)
                need_c = dp.dp_clip_accumulate_embedding_workspace_bytes(N, layer.V)
            elif isinstance(layer, W.LayerNorm):
                lb.gW = torch.empty((N, layer.D), **f32)
                lb.gb = torch.empty((N, layer.D), **f32)
                need_g = dp.dp_grad_sample_layernorm_workspace_bytes(N, layer.T, layer.D)
            elif isinstance(layer, W.GroupNorm):
                lb.gW = torch.empty((N, layer.C), **f32)
                lb.gb = torch.empty((N, layer.C), **f32)
                need_g = dp.dp_grad_sample_groupnorm_workspace_bytes(N, layer.C, layer.P)
            # each layer has its own scratch, so its calls may run concurrently with other layers'
            lb.ws = torch.empty(max(need_g, 256), dtype=torch.uint8, device=self.device)
            lb.ws_clip = torch.empty(max(need_c, 256), dtype=torch.uint8, device=self.device)
            self.layers.append(lb)
        self.sqnorm = torch.empty((len(self.layers), N), **f32)
        for i, lb in enumerate(self.layers):
            if isinstance(lb.layer, W.LSTMRecurrence):
                self.sqnorm[i].zero_()            # no parameters: its row stays zero
        self.norm = torch.empty(N, **f32)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.params = wl.param_tensors()
        self.S: Dict[str, object] = {}
        self.out: Dict[str, object] = {}
        for name, shape in self.params:
            self.S[name] = torch.empty(shape, **f32)
            self.out[name] = torch.empty(shape, **f32)
        # the fused Linear clipped sums (B^T diag(c) A) run as one grouped call
        self.fused_linear = [i for i, lb in enumerate(self.layers)
                             if isinstance(lb.layer, W.Linear) and lb.clip_mode == "fused"]
        ents = []
        for i in self.fused_linear:
            lb = self.layers[i]
            L = lb.layer
            # the bias sums are column reductions of the stored per-sample bias
            # gradients (N x d_out values) in the grouped clip/noise call,
            # unless the layer's gradients are not formed (ghost norms)
            sumb = self.S[L.name + ".bias"] if (lb.ghost and L.bias) else None
            ents.append((lb.A, lb.B, L.T, L.d_in, L.d_out, self.scale, self.S[L.name + ".weight"], sumb))
        self.linear_items = dp.make_linear_clips(ents)
        need = dp.dp_clip_accumulate_linear_many_workspace_bytes(self.linear_items, len(ents), self.dt, N)
        self.ws_linear = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        # the grouped clip/noise call: per-sample grads for column-reduced tensors
        entries = []
        for pidx, (name, shape) in enumerate(self.params):
            entries.append((self._grad_for(name), self.S[name], self.out[name], int(np.prod(shape)), pidx))
        self.group = dp.make_params(entries)
        self.group_count = len(entries)
        # virtual steps: running sums, a group that only accumulates and one
        # that accumulates and forms the output
        self.acc: Dict[str, object] = {}
        if self.virtual_batches > 1:
            for name, shape in self.params:
                self.acc[name] = torch.zeros(shape, **f32)
            ents_acc, ents_emit = [], []
            for (g, s_, o, numel, pidx), (name, _) in zip(entries, self.params):
                ents_acc.append((g, s_, None, numel, pidx, self.acc[name]))
                ents_emit.append((g, s_, o, numel, pidx, self.acc[name]))
            self.group_acc = dp.make_params(ents_acc)
            self.group_emit = dp.make_params(ents_emit)
        # the norms are computed inside the clip/noise launch unless a fused
        # clipped sum (which needs them) runs before it
        self.fold_norms = not self.fused_linear and not any(isinstance(lb.layer, W.Embedding)
                                                              for lb in self.layers)
        need = dp.dp_norms_clip_noise_workspace_bytes(self.group, self.group_count, N)
        self.ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        # Linear (T = 1) and small Conv2d layers: per-sample grads in one grouped launch
        self.grad_group: List[int] = []
        items = [self._grad_item(i) for i in range(len(self.layers))]
        cand = [i for i, it in enumerate(items) if it is not None]
        if cand:
            arr = dp.make_layer_grads([items[i] for i in cand])
            grouped = [i for k, i in enumerate(cand) if dp.dp_grad_sample_many_grouped(arr, k, self.dt, N)]
            if len(grouped) >= 2:
                self.grad_group = grouped
                self.group_items = dp.make_layer_grads([items[i] for i in grouped])
                need = dp.dp_grad_sample_many_workspace_bytes(self.group_items, len(grouped), self.dt, N)
                self.ws_group = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        # LayerNorm layers: one grouped call over all of them
        self.lns = [i for i, lb in enumerate(self.layers) if isinstance(lb.layer, W.LayerNorm)]
        if self.lns:
            self.ln_items = dp.make_layernorm_layers(
                [(lb.A, lb.B, lb.layer.T, lb.layer.D, self.scale, lb.gW, lb.gb, self.sqnorm[i])
                 for i, lb in ((i, self.layers[i]) for i in self.lns)])
            need = dp.dp_grad_sample_layernorm_many_workspace_bytes(self.ln_items, len(self.lns), N, self.dt)
            self.ws_lns = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        # ghost-norm Linear layers: one grouped call over all of them
        self.ghost = [i for i, lb in enumerate(self.layers) if lb.ghost]
        if self.ghost:
            self.ghost_items = dp.make_ghost_layers(
                [(lb.A, lb.B, lb.layer.T, lb.layer.d_in, lb.layer.d_out, self.scale, lb.layer.bias, self.sqnorm[i])
                 for i, lb in ((i, self.layers[i]) for i in self.ghost)])
            need = dp.dp_ghost_norm_linear_many_workspace_bytes(self.ghost_items, len(self.ghost), N)
            self.ws_ghost = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        self.step_dev = torch.zeros(1, dtype=torch.int64, device=self.device)
        self.graph = None
        self.graph_parallel = None
        self.steps_per_replay = 1
        self._side = None

    def _grad_for(self, pname: str):
        """The per-sample grad buffer of a parameter if it is column-reduced, else None."""
        lname, key = pname.rsplit(".", 1)
        for lb in self.layers:
            if lb.layer.name != lname:
                continue
            if isinstance(lb.layer, W.Embedding):
                return None
            if isinstance(lb.layer, W.Linear) and lb.clip_mode == "fused" and (key == "weight" or lb.ghost):
                return None
            return lb.gW if key == "weight" else lb.gb
        raise KeyError(pname)

    def _grad_item(self, i: int):
        """Layer i as a dp_layer_grad entry (Linear and Conv2d only), else None."""
        lb = self.layers[i]
        L = lb.layer
        sq = self.sqnorm[i]
        if isinstance(L, W.Linear):
            if lb.ghost:
                return None
            return dp.linear_grad_item(lb.A, lb.B, L.T, L.d_in, L.d_out, self.scale, lb.gW, lb.gb, sq)
        if isinstance(L, W.Conv2d):
            ho, wo = L.out_hw
            return dp.conv2d_grad_item(lb.A, lb.B, L.c_in, L.h, L.w, L.c_out, ho, wo, L.k[0], L.k[1], L.stride[0],
                                       L.stride[1], L.pad[0], L.pad[1], self.scale, lb.gW, lb.gb, sq)
        return None

    def recurrence_calls(self) -> List[str]:
        """Backward-through-time calls, which the gradient calls of the layers they feed wait for."""
        return ["grad:" + lb.layer.name for lb in self.layers if isinstance(lb.layer, W.LSTMRecurrence)]

    def grad_calls(self) -> List[str]:
        """The per-sample-gradient calls of a step, in order (after the recurrences)."""
        calls = ["grad:group"] if self.grad_group else []
        calls += ["grad:ghost"] if self.ghost else []
        calls += ["grad:lns"] if self.lns else []
        return calls + ["grad:" + lb.layer.name for i, lb in enumerate(self.layers)
                        if i not in self.grad_group and not lb.ghost and i not in self.lns
                        and not isinstance(lb.layer, W.LSTMRecurrence)]

    # ------------------------------------------------------------------ pieces
    def grad_group_call(self, stream=None):
        """The grouped layers' per-sample gradients in one launch."""
        dp.dp_grad_sample_many(self.group_items, len(self.grad_group), self.dt, self.N, self.status, self.ws_group,
                               stream)

    def ghost_call(self, stream=None):
        """The ghost-norm layers' per-sample squared norms in one grouped call."""
        dp.dp_ghost_norm_linear_many(self.ghost_items, len(self.ghost), self.dt, self.N, self.status, self.ws_ghost,
                                     stream)

    def layernorm_call(self, stream=None):
        """The LayerNorm layers' affine gradients in one grouped call."""
        dp.dp_grad_sample_layernorm_many(self.ln_items, len(self.lns), self.dt, self.N, self.status, self.ws_lns,
                                         stream)

    def grad_sample(self, i: int, stream=None):
        lb = self.layers[i]
        layer = lb.layer
        N, s, sq = self.N, self.scale, self.sqnorm[i]
        if isinstance(layer, W.LSTMRecurrence):
            a = lb.aux
            dp.dp_lstm_backward(a["gates"], a["c"], a["W_hh"], None, a["dh_last"], N, layer.T, layer.H, lb.B,
                                self.status, stream)
        elif isinstance(layer, W.Linear) and lb.ghost:
            raise KeyError("ghost-norm layer %s runs in the grouped call grad:ghost" % layer.name)
        elif isinstance(layer, W.Linear):
            dp.dp_grad_sample_linear(lb.A, lb.B, self.dt, N, layer.T, layer.d_in, layer.d_out, s, lb.gW, lb.gb,
                                     sq, self.status, lb.ws, stream)
        elif isinstance(layer, W.Conv2d):
            ho, wo = layer.out_hw
            dp.dp_grad_sample_conv2d(lb.A, lb.B, self.dt, N, layer.c_in, layer.h, layer.w, layer.c_out, ho, wo,
                                     layer.k[0], layer.k[1], layer.stride[0], layer.stride[1], layer.pad[0],
                                     layer.pad[1], 1, 1, 1, s, lb.gW, lb.gb, sq, self.status, lb.ws, stream)
        elif isinstance(layer, W.Embedding):
            dp.dp_grad_sample_embedding(lb.ids, lb.B, self.dt, N, layer.T, layer.V, layer.D, s, lb.row_ptr,
                                        lb.uniq, lb.rows, N * layer.T, sq, self.status, lb.ws, stream)
        elif isinstance(layer, W.LayerNorm):
            dp.dp_grad_sample_layernorm(lb.A, lb.B, self.dt, N, layer.T, layer.D, s, lb.gW, lb.gb, sq,
                                        self.status, lb.ws, stream)
        elif isinstance(layer, W.GroupNorm):
            dp.dp_grad_sample_groupnorm(lb.A, lb.B, self.dt, N, layer.C, layer.P, s, lb.gW, lb.gb, sq,
                                        self.status, lb.ws, stream)

    def norms(self, stream=None):
        if self.n_active is not None:
            dp.dp_per_sample_norms_active(self.sqnorm, len(self.layers), self.N, self.n_active, self.norm,
                                          self.status, stream)
        else:
            dp.dp_per_sample_norms(self.sqnorm, len(self.layers), self.N, self.norm, self.status, stream)

    def set_active(self, n: int):
        """The size of the variable batch (rows 0..n-1 of the step's N), written
        to device memory on the current stream (not inside a captured graph)."""
        if self.n_active is None:
            raise RuntimeError("set_active needs a DPStep built with variable_batch=True")
        if not 0 <= int(n) <= self.N:
            raise ValueError("active batch size %d outside [0, %d]" % (n, self.N))
        self.n_active.fill_(int(n))

    def linear_clip_sums(self, stream=None):
        """The fused Linear layers' clipped sums, in one grouped call."""
        if self.fused_linear:
            dp.dp_clip_accumulate_linear_many(self.linear_items, len(self.fused_linear), self.dt, self.N, self.norm,
                                              self.C, self.status, self.ws_linear, stream)

    def fused_clip_sum(self, i: int, stream=None):
        """Clipped sums formed without reading per-sample grads (Embedding)."""
        lb = self.layers[i]
        layer = lb.layer
        name = layer.name
        if isinstance(layer, W.Embedding):
            dp.dp_clip_accumulate_embedding(lb.row_ptr, lb.uniq, lb.rows, lb.uniq.shape[0], self.norm, self.C,
                                            self.N, layer.V, layer.D, self.S[name + ".weight"], self.status,
                                            lb.ws_clip, stream)

    def clip_noise(self, step: int, step_dev=None, stream=None, emit: bool = True):
        """Clipped sums, noise and division of every tensor (and the norms, when folded) in one launch.
        With virtual steps the sums go into the running sums, and the output
        is formed only when emit is set (the logical batch's last physical batch)."""
        group = self.group if self.virtual_batches == 1 else (self.group_emit if emit else self.group_acc)
        if self.sigma_tab is not None:
            dp.dp_norms_clip_noise_sched(self.sqnorm if self.fold_norms else None, len(self.layers), group,
                                         self.group_count, self.N, self.norm, self.C, self.seed, step, step_dev,
                                         self.sigma_tab, self.denom, self.status, self.ws, stream,
                                         n_active=self.n_active)
        else:
            dp.dp_norms_clip_noise(self.sqnorm if self.fold_norms else None, len(self.layers), group,
                                   self.group_count, self.N, self.norm, self.C, self.seed, step, step_dev,
                                   self.sigma, self.denom, self.status, self.ws, stream)

    def reset_running_sums(self):
        """Zero the virtual step's running sums (a fill kernel, capturable)."""
        for t in self.acc.values():
            t.zero_()

    def call(self, name: str, step: int = 0, stream=None):
        """Enqueue one named call of the step ("grad:<layer>", "norms", "clip:<layer>", "clip+noise")."""
        if name == "norms":
            return None if self.fold_norms else self.norms(stream)
        if name == "clip+noise":
            return self.clip_noise(step, None, stream)
        if name == "clip:linears":
            return self.linear_clip_sums(stream)
        if name == "grad:group":
            return self.grad_group_call(stream)
        if name == "grad:ghost":
            return self.ghost_call(stream)
        if name == "grad:lns":
            return self.layernorm_call(stream)
        kind, lname = name.split(":", 1)
        i = next(k for k, lb in enumerate(self.layers) if lb.layer.name == lname)
        if kind == "grad":
            return self.grad_sample(i, stream)
        if kind == "clip":
            return self.fused_clip_sum(i, stream)
        raise KeyError(name)

    def _fork(self, n):
        torch = _torch()
        if self._side is None or len(self._side) < n:
            self._side = [torch.cuda.Stream(self.device) for _ in range(n)]
        return self._side[:n]

    # ------------------------------------------------------------------ whole step
    def run(self, step: int = 0, stream=None, mark: Optional[Callable[[str, str], None]] = None, step_dev=None,
            parallel: bool = False, advance: int = 0, clear_status: bool = True, reset: bool = True,
            emit: bool = True):
        """Enqueue one whole step; nothing is synchronized here.

        parallel: the layers' per-sample-gradient calls (independent of each
        other) and the fused clipped sums run on side streams forked from and
        joined back into the current stream.  advance: if nonzero, also
        enqueue dp_step_advance(step_dev, advance), in a branch ahead of the
        noise.
        clear_status: zero the status word first (a captured step leaves it
        alone, so flags accumulate over replays until the caller clears it).
        reset, emit (virtual steps only): zero the running sums first (the
        logical batch's first physical batch); form the output (its last)."""
        torch = _torch()
        if clear_status:
            self.status.zero_()
        if self.virtual_batches > 1 and reset:
            self.reset_running_sums()
        if not parallel:
            if advance:
                dp.dp_step_advance(step_dev, advance, stream)
            for name in self.recurrence_calls() + self.grad_calls():
                if mark: mark(name, "start")
                self.call(name, step, stream)
                if mark: mark(name, "end")
            if not self.fold_norms:
                if mark: mark("norms", "start")
                self.norms(stream)
                if mark: mark("norms", "end")
            if self.fused_linear:
                if mark: mark("clip:linears", "start")
                self.linear_clip_sums(stream)
                if mark: mark("clip:linears", "end")
            for i, lb in enumerate(self.layers):
                if isinstance(lb.layer, W.Embedding):
                    if mark: mark("clip:" + lb.layer.name, "start")
                    self.fused_clip_sum(i, stream)
                    if mark: mark("clip:" + lb.layer.name, "end")
            if mark: mark("clip+noise", "start")
            self.clip_noise(step, step_dev, stream, emit)
            if mark: mark("clip+noise", "end")
            return
        main = torch.cuda.current_stream(self.device)
        side = self._fork(len(self.layers) + 1)
        for name in self.recurrence_calls():      # before the branches that read their output
            self.call(name, step)
        for k, name in enumerate(self.grad_calls()):
            side[k].wait_stream(main)
            with torch.cuda.stream(side[k]):
                self.call(name, step)
        if advance:
            side[-1].wait_stream(main)
            with torch.cuda.stream(side[-1]):
                dp.dp_step_advance(step_dev, advance)
        for s_ in side:
            main.wait_stream(s_)
        if not self.fold_norms:
            self.norms()
        fused = [i for i, lb in enumerate(self.layers) if isinstance(lb.layer, W.Embedding)]
        for k, i in enumerate(fused):
            side[k].wait_stream(main)
            with torch.cuda.stream(side[k]):
                self.fused_clip_sum(i)
        k_lin = len(fused)
        if self.fused_linear:
            side[k_lin].wait_stream(main)
            with torch.cuda.stream(side[k_lin]):
                self.linear_clip_sums()
        for k in range(len(fused) + (1 if self.fused_linear else 0)):
            main.wait_stream(side[k])
        self.clip_noise(step, step_dev, emit=emit)

    def capture(self, first_step: int = 0, parallel: Optional[bool] = None, steps_per_replay: int = 1):
        """Capture steps as a HIP graph; replay j runs steps first_step + j*r
        .. first_step + j*r + r - 1 (r = steps_per_replay).

        The graph advances its own device step counter by r at the start of
        each replay (in a branch that runs before the noise); step k of the
        replay uses step_dev + k.  Nothing is re-recorded between replays,
        and step_dev holds the first step of the last replay.
        parallel: the layers' calls as parallel branches of the graph (True),
        or one chain (False); None captures both, times a few replays of
        each and keeps the faster (branches pay off when the layers' kernels
        are long enough to overlap; for short kernels the single chain has
        less scheduling overhead).  Branches are supported with one step per
        replay only (a branch graph of two transformer-block steps ended the
        process inside the graph launch, cause not found): True with
        steps_per_replay > 1 raises ValueError, and None compares the chain
        at steps_per_replay with branches at one step per replay.
        steps_per_replay: whole steps recorded back to back in the graph, so
        that one replay launch covers several steps (each still a full pass
        over the batch, with its own step number)."""
        torch = _torch()
        if parallel is True and steps_per_replay > 1:
            raise ValueError("graph branches are supported with one step per replay only")
        if parallel is None:
            # the chain at steps_per_replay steps per replay against branches
            # at one, per step; the faster is kept (with branches the graph
            # then holds one step, and self.steps_per_replay says so)
            import time

            def per_step(par, r):
                self.capture(first_step, par, r)
                for _ in range(3):
                    self.replay()
                torch.cuda.synchronize(self.device)
                n = max(40 // r, 4)
                t0 = time.perf_counter()
                for _ in range(n):
                    self.replay()
                torch.cuda.synchronize(self.device)
                return (time.perf_counter() - t0) / (n * r)
            cands = [(False, steps_per_replay), (True, 1)]
            best = min(cands, key=lambda c: per_step(*c))
            return self.capture(first_step, best[0], best[1])
        side = torch.cuda.Stream(self.device)
        side.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(side):
            self.run(step=0, parallel=parallel)          # warm up outside the capture
        torch.cuda.current_stream(self.device).wait_stream(side)
        torch.cuda.synchronize(self.device)
        g = torch.cuda.CUDAGraph()
        K = self.virtual_batches
        with torch.cuda.graph(g):
            for i in range(steps_per_replay):
                for k in range(K):
                    # virtual steps: K physical batches (here the resident inputs each time) of
                    # logical step i; the counter moves once per replay
                    self.run(step=i, step_dev=self.step_dev, parallel=parallel,
                             advance=steps_per_replay if (i == 0 and k == 0) else 0,
                             clear_status=False, reset=(k == 0), emit=(k == K - 1))
        torch.cuda.synchronize(self.device)
        self.step_dev.fill_(first_step - steps_per_replay)    # advanced to first_step by the first replay
        self.graph = g
        self.graph_parallel = parallel
        self.steps_per_replay = steps_per_replay
        return g

    def load_inputs(self, inputs: List[W.LayerInputs]):
        """Copy another physical batch's inputs (same shapes) into the step's device buffers."""
        torch = _torch()
        for lb, li in zip(self.layers, inputs):
            if li.A is not None:
                lb.A.copy_(to_device(li.A, self.wl.dtype, self.device))
            if li.aux is not None:
                for k, v in li.aux.items():
                    lb.aux[k].copy_(to_device(v, W.F32, self.device))
            if li.B is not None:
                lb.B.copy_(to_device(li.B, self.wl.dtype, self.device))
            if li.ids is not None:
                lb.ids.copy_(to_device(li.ids, "", self.device))

    def run_virtual(self, batches: List[List[W.LayerInputs]], step: int = 0):
        """One logical step over the physical batches `batches` (each with this step's N samples), eagerly."""
        if len(batches) != self.virtual_batches:
            raise ValueError("expected %d physical batches" % self.virtual_batches)
        for k, inputs in enumerate(batches):
            self.load_inputs(inputs)
            self.run(step=step, clear_status=(k == 0), reset=(k == 0), emit=(k == len(batches) - 1))

    def replay(self):
        self.graph.replay()

    def results(self) -> Dict[str, object]:
        """Copy everything back to host numpy arrays (synchronizes)."""
        torch = _torch()
        torch.cuda.synchronize(self.device)
        res = {"grads": [], "sq_layers": self.sqnorm.cpu().numpy(), "norm": self.norm.cpu().numpy(),
               "S": {k: v.cpu().numpy() for k, v in self.S.items()},
               "out": {k: v.cpu().numpy() for k, v in self.out.items()},
               "status": int(self.status.cpu().item()),
               "acc": {k: v.cpu().numpy() for k, v in self.acc.items()}}
        res["derived"] = {lb.layer.name: lb.B.cpu().numpy() for lb in self.layers
                          if isinstance(lb.layer, W.LSTMRecurrence)}
        for lb in self.layers:
            if isinstance(lb.layer, W.LSTMRecurrence):
                res["grads"].append({})            # no parameters of its own
            elif isinstance(lb.layer, W.Embedding):
                rp = lb.row_ptr.cpu().numpy()
                nnz = int(rp[-1])
                res["grads"].append({"csr": (rp, lb.uniq[:nnz].cpu().numpy(), lb.rows[:nnz].cpu().numpy())})
            elif lb.gW is None:
                res["grads"].append({})            # ghost norm: no per-sample gradient formed
            else:
                g = {"weight": lb.gW.cpu().numpy()}
                if lb.gb is not None:
                    g["bias"] = lb.gb.cpu().numpy()
                res["grads"].append(g)
        return res
