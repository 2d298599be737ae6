"""Seeded synthetic inputs for the DP-SGD gradient step.

This module only draws numbers.  It holds none of the step's arithmetic, so the
HIP library and the oracle can both be fed from it without sharing any code of
the method itself.

Each workload is a list of layers in forward order.  For every layer it draws
the activation that enters the layer (``A``; for an embedding the token ids)
and the backprop at the layer's output (``B``), the two tensors the paper's
vectorized method starts from (appendix "Vectorized Computation": activations
are kept by forward hooks, highway gradients by backward hooks).

Streams: ``numpy.random.default_rng([workload_id, tensor_id])`` (a PCG64 seed
sequence), one independent stream per tensor, numbered in forward layer order
with a layer's activation before its backprop.  bf16 tensors are drawn in fp32
and rounded to nearest-even on the host; both sides then consume the same
bf16 bits.

Stand-ins: the paper trains on MNIST, CIFAR-10 and IMDb (section 3.1.2).  No
dataset item is used; the activations and backprops below have the shapes of
those networks' layers and simple distributions (N(0,1), post-ReLU
max(0, N(0,1)), backprops N(0,1)/batch, token ids Zipf(1.1)).

One workload (``text_lstm_bptt``) stores what an LSTM's forward pass keeps:
its gate activations, cell states and hidden states over the sequence, from
a forward over the embedded tokens with randomly initialised weights (the
model's own forward, run here in numpy; the DP step starts after it).  Its
gate backprop is not drawn: the step derives it by the backward through time.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class Linear:
    """A Linear layer y = x W^T + b applied over a sequence of T positions.

    ``A`` is [N, T, d_in], ``B`` is [N, T, d_out]; T == 1 is the plain
    (non-sequence) layer and is stored as [N, d_in] / [N, d_out].
    """
    name: str
    d_in: int
    d_out: int
    T: int = 1
    bias: bool = True
    act: str = "normal"          # A: normal | relu | tanh_prev | tanh_last | embed | lstm_x | lstm_hprev | lstm_hlast
    bshare: Optional[str] = None  # name of a layer whose B this layer reuses (LSTM W_ih / W_hh)
    bsource: Optional[str] = None  # name of an LSTMRecurrence whose derived gate backprop is this layer's B

    @property
    def n_params(self) -> int:
        return self.d_out * self.d_in + (self.d_out if self.bias else 0)


@dataclass(frozen=True)
class Conv2d:
    """Conv2d (groups=1, dilation=1) on [N, Cin, H, W] giving [N, Cout, Ho, Wo]."""
    name: str
    c_in: int
    c_out: int
    h: int
    w: int
    k: Tuple[int, int]
    stride: Tuple[int, int] = (1, 1)
    pad: Tuple[int, int] = (0, 0)
    bias: bool = True
    act: str = "relu"

    @property
    def out_hw(self) -> Tuple[int, int]:
        ho = (self.h + 2 * self.pad[0] - self.k[0]) // self.stride[0] + 1
        wo = (self.w + 2 * self.pad[1] - self.k[1]) // self.stride[1] + 1
        return ho, wo

    @property
    def n_params(self) -> int:
        return self.c_out * self.c_in * self.k[0] * self.k[1] + (self.c_out if self.bias else 0)


@dataclass(frozen=True)
class Embedding:
    """Embedding lookup: token ids [N, T] into a [V, D] table."""
    name: str
    V: int
    D: int
    T: int
    zipf_s: float = 1.1
    truncate: bool = False  # False: ids clipped to V-1; True: ids redrawn (rejection) until < V

    @property
    def n_params(self) -> int:
        return self.V * self.D


@dataclass(frozen=True)
class LayerNorm:
    """LayerNorm's elementwise affine y = g * xhat + b over D features, T positions."""
    name: str
    D: int
    T: int
    @property
    def n_params(self) -> int:
        return 2 * self.D


@dataclass(frozen=True)
class GroupNorm:
    """GroupNorm's (or InstanceNorm's) per-channel affine y = g[c] * xhat + b[c]
    over C channels of P spatial positions each."""
    name: str
    C: int
    P: int
    @property
    def n_params(self) -> int:
        return 2 * self.C


@dataclass(frozen=True)
class LSTMRecurrence:
    """The backward through time of an LSTM layer (input D, hidden H, T steps).

    It has no parameters of its own: the LSTM's weights are the Linear layers
    that name it as ``bsource`` (W_ih over x_t, W_hh over h_{t-1}, each with
    its bias), and their per-sample gradients take the gate backprop this
    layer derives, from the stored gate activations and cell states and the
    loss gradient arriving at the last hidden state, as B."""
    name: str
    D: int
    H: int
    T: int

    @property
    def n_params(self) -> int:
        return 0


@dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    N: int
    dtype: str
    C: float
    sigma: float
    layers: Tuple
    seed: int = 0
    scale: float = 1.0
    notes: str = ""

    @property
    def n_params(self) -> int:
        return sum(l.n_params for l in self.layers)

    def param_tensors(self) -> List[Tuple[str, Tuple[int, ...]]]:
        """(name, shape) of every parameter tensor, in the order noise indices follow."""
        out = []
        for l in self.layers:
            if isinstance(l, Linear):
                out.append((l.name + ".weight", (l.d_out, l.d_in)))
                if l.bias:
                    out.append((l.name + ".bias", (l.d_out,)))
            elif isinstance(l, Conv2d):
                out.append((l.name + ".weight", (l.c_out, l.c_in, l.k[0], l.k[1])))
                if l.bias:
                    out.append((l.name + ".bias", (l.c_out,)))
            elif isinstance(l, Embedding):
                out.append((l.name + ".weight", (l.V, l.D)))
            elif isinstance(l, LayerNorm):
                out.append((l.name + ".weight", (l.D,)))
                out.append((l.name + ".bias", (l.D,)))
            elif isinstance(l, GroupNorm):
                out.append((l.name + ".weight", (l.C,)))
                out.append((l.name + ".bias", (l.C,)))
        return out


def _build_workloads() -> Dict[str, Workload]:
    w = {}
    # A single Linear 64 -> 16 with bias, batch 32.
    w["linear_tiny"] = Workload(
        0, "linear_tiny", N=32, dtype=F32, C=1.0, sigma=1.0,
        layers=(Linear("fc", 64, 16, act="normal"),))
    # MNIST-shaped CNN (26,010 parameters, the count given in section 3.1.2).
    # A 2x2 stride-1 pool after each conv gives conv2 a 13x13 input and fc1 512 inputs.
    w["mnist_cnn"] = Workload(
        1, "mnist_cnn", N=256, dtype=F32, C=1.0, sigma=1.1,
        layers=(Conv2d("conv1", 1, 16, 28, 28, (8, 8), (2, 2), (3, 3)),
                Conv2d("conv2", 16, 32, 13, 13, (4, 4), (2, 2), (0, 0)),
                Linear("fc1", 512, 32, act="relu"),
                Linear("fc2", 32, 10, act="relu")))
    # CIFAR-shaped CNN, batch 512.
    w["cifar_cnn"] = Workload(
        2, "cifar_cnn", N=512, dtype=F32, C=1.5, sigma=1.5,
        layers=(Conv2d("c1", 3, 32, 32, 32, (3, 3), (1, 1), (1, 1)),
                Conv2d("c2", 32, 64, 32, 32, (3, 3), (1, 1), (1, 1)),
                Conv2d("c3", 64, 64, 16, 16, (3, 3), (1, 1), (1, 1)),
                Conv2d("c4", 64, 128, 16, 16, (3, 3), (1, 1), (1, 1)),
                Conv2d("c5", 128, 128, 8, 8, (3, 3), (1, 1), (1, 1)),
                Conv2d("c6", 128, 256, 8, 8, (3, 3), (1, 1), (1, 1)),
                Linear("fc", 4096, 10, act="relu")))
    # Text LSTM on IMDb-shaped input (1,081,002 parameters, section 3.1.2).
    w["text_lstm"] = Workload(
        3, "text_lstm", N=64, dtype=F32, C=1.0, sigma=1.0,
        layers=(Embedding("emb", 10000, 100, 256),
                Linear("lstm_ih", 100, 400, T=256, act="embed"),
                Linear("lstm_hh", 100, 400, T=256, act="tanh_prev", bshare="lstm_ih"),
                Linear("fc", 100, 2, act="tanh_last")))
    # The text LSTM with its gate backprop derived by the backward through time
    # from a forward pass's stored activations (same shapes and parameters).
    w["text_lstm_bptt"] = Workload(
        6, "text_lstm_bptt", N=64, dtype=F32, C=1.0, sigma=1.0,
        layers=(Embedding("emb", 10000, 100, 256),
                LSTMRecurrence("lstm", 100, 100, 256),
                Linear("lstm_ih", 100, 400, T=256, act="lstm_x", bsource="lstm"),
                Linear("lstm_hh", 100, 400, T=256, act="lstm_hprev", bsource="lstm"),
                Linear("fc", 100, 2, act="lstm_hlast")))
    # Transformer encoder block, bf16 activations/backprops.
    w["transformer_block"] = Workload(
        4, "transformer_block", N=32, dtype=BF16, C=1.0, sigma=0.8,
        layers=(Linear("wq", 768, 768, T=128), Linear("wk", 768, 768, T=128),
                Linear("wv", 768, 768, T=128), Linear("wo", 768, 768, T=128),
                LayerNorm("ln1", 768, 128),
                Linear("ffn1", 768, 3072, T=128), Linear("ffn2", 3072, 768, T=128),
                LayerNorm("ln2", 768, 128)))
    # The CIFAR-shaped CNN with a GroupNorm after each convolution (the
    # normalization layers Opacus supports per sample), batch 512.
    w["cifar_gn"] = Workload(
        5, "cifar_gn", N=512, dtype=F32, C=1.5, sigma=1.5,
        layers=(Conv2d("c1", 3, 32, 32, 32, (3, 3), (1, 1), (1, 1)), GroupNorm("g1", 32, 1024),
                Conv2d("c2", 32, 64, 32, 32, (3, 3), (1, 1), (1, 1)), GroupNorm("g2", 64, 1024),
                Conv2d("c3", 64, 64, 16, 16, (3, 3), (1, 1), (1, 1)), GroupNorm("g3", 64, 256),
                Conv2d("c4", 64, 128, 16, 16, (3, 3), (1, 1), (1, 1)), GroupNorm("g4", 128, 256),
                Conv2d("c5", 128, 128, 8, 8, (3, 3), (1, 1), (1, 1)), GroupNorm("g5", 128, 64),
                Conv2d("c6", 128, 256, 8, 8, (3, 3), (1, 1), (1, 1)), GroupNorm("g6", 256, 64),
                Linear("fc", 4096, 10, act="relu")))
    return w


WORKLOADS: Dict[str, Workload] = _build_workloads()
WORKLOAD_ORDER = ["linear_tiny", "mnist_cnn", "cifar_cnn", "text_lstm", "transformer_block", "cifar_gn",
                  "text_lstm_bptt"]


def get(name: str) -> Workload:
    return WORKLOADS[name]


def _rng(wid: int, tid: int) -> np.random.Generator:
    return np.random.default_rng([wid, tid])


def _normal(rng, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def _zipf_ids(rng, shape, V: int, s: float, truncate: bool) -> np.ndarray:
    k = rng.zipf(s, size=shape).astype(np.int64)
    if truncate:
        bad = k > V
        while bad.any():
            k[bad] = rng.zipf(s, size=int(bad.sum()))
            bad = k > V
        return k - 1
    return np.minimum(k, V) - 1


@dataclass
class LayerInputs:
    layer: object
    A: Optional[np.ndarray] = None     # activation (fp32 array; bf16 workloads round later)
    B: Optional[np.ndarray] = None     # backprop at the layer output (None: derived by the step)
    ids: Optional[np.ndarray] = None   # int64 token ids (embedding)
    aux: Optional[Dict[str, np.ndarray]] = None   # LSTMRecurrence: gates, c, W_hh, dh_last


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def lstm_forward_activations(x: np.ndarray, W_ih, W_hh, b_ih, b_hh):
    """The stored activations of an LSTM forward over x [N, T, D] (gate order
    i, f, g, o, zero initial state), in float64: gates after their
    nonlinearities [N, T, 4H], cell states and hidden states [N, T, H]."""
    N, T, _ = x.shape
    H = W_hh.shape[1]
    gates = np.empty((N, T, 4 * H)); c = np.empty((N, T, H)); h = np.empty((N, T, H))
    hp = np.zeros((N, H)); cp = np.zeros((N, H))
    for t in range(T):
        z = x[:, t] @ W_ih.T + b_ih + hp @ W_hh.T + b_hh
        i, f, g, o = _sigmoid(z[:, :H]), _sigmoid(z[:, H:2 * H]), np.tanh(z[:, 2 * H:3 * H]), _sigmoid(z[:, 3 * H:])
        cp = f * cp + i * g
        hp = o * np.tanh(cp)
        gates[:, t] = np.concatenate([i, f, g, o], axis=1)
        c[:, t] = cp
        h[:, t] = hp
    return gates, c, h


def make_inputs(wl: Workload, n: Optional[int] = None) -> List[LayerInputs]:
    """Draw every layer's inputs for workload ``wl``.

    ``n`` overrides the batch size (a prefix-free redraw, used for small
    parity cases of the same shapes).  Returned arrays are float32 (ids int64);
    use :func:`to_bf16_bits` / :func:`torch_inputs` for the bf16 workloads.
    """
    N = wl.N if n is None else int(n)
    out: List[LayerInputs] = []
    by_name: Dict[str, LayerInputs] = {}
    tid = 0
    emb_table = None
    emb_ids = None
    lstm_hidden = None
    lstm_fwd = None           # (x, h) of an LSTMRecurrence's forward pass
    for layer in wl.layers:
        li = LayerInputs(layer)
        if isinstance(layer, Conv2d):
            rA = _rng(wl.wid, tid); tid += 1
            rB = _rng(wl.wid, tid); tid += 1
            ho, wo = layer.out_hw
            a = _normal(rA, (N, layer.c_in, layer.h, layer.w))
            if layer.act == "relu":
                np.maximum(a, 0, out=a)
            li.A = a
            li.B = _normal(rB, (N, layer.c_out, ho, wo)) / np.float32(wl.N)
        elif isinstance(layer, Linear):
            rA = _rng(wl.wid, tid); tid += 1
            rB = _rng(wl.wid, tid); tid += 1
            shapeA = (N, layer.d_in) if layer.T == 1 else (N, layer.T, layer.d_in)
            shapeB = (N, layer.d_out) if layer.T == 1 else (N, layer.T, layer.d_out)
            if layer.act == "normal":
                a = _normal(rA, shapeA)
            elif layer.act == "relu":
                a = np.maximum(_normal(rA, shapeA), 0)
            elif layer.act == "embed":
                # LSTM input x_t = E[ids_t], E ~ N(0,1) (nn.Embedding's default init).
                if emb_table is None:
                    emb_table = _normal(rA, (by_name_emb(wl).V, by_name_emb(wl).D))
                a = emb_table[emb_ids]
            elif layer.act in ("lstm_x", "lstm_hprev", "lstm_hlast"):
                x, h = lstm_fwd
                if layer.act == "lstm_x":
                    a = x
                elif layer.act == "lstm_hprev":
                    a = np.zeros_like(h)
                    a[:, 1:, :] = h[:, :-1, :]
                else:
                    a = np.ascontiguousarray(h[:, -1, :])
            elif layer.act in ("tanh_prev", "tanh_last"):
                if lstm_hidden is None:
                    T = layer.T if layer.T > 1 else max(l.T for l in wl.layers if isinstance(l, Linear))
                    lstm_hidden = np.tanh(_normal(rA, (N, T, layer.d_in)))
                if layer.act == "tanh_prev":
                    a = np.zeros_like(lstm_hidden)
                    a[:, 1:, :] = lstm_hidden[:, :-1, :]
                else:
                    a = np.ascontiguousarray(lstm_hidden[:, -1, :])
            else:
                raise ValueError(layer.act)
            li.A = np.ascontiguousarray(a, dtype=np.float32)
            if layer.bsource is not None:
                li.B = None                      # derived by the step (backward through time)
            elif layer.bshare is not None:
                li.B = by_name[layer.bshare].B
            else:
                li.B = _normal(rB, shapeB) / np.float32(wl.N)
        elif isinstance(layer, Embedding):
            rA = _rng(wl.wid, tid); tid += 1
            rB = _rng(wl.wid, tid); tid += 1
            li.ids = _zipf_ids(rA, (N, layer.T), layer.V, layer.zipf_s, layer.truncate)
            emb_ids = li.ids
            li.B = _normal(rB, (N, layer.T, layer.D)) / np.float32(wl.N)
        elif isinstance(layer, LSTMRecurrence):
            # the embedding table, the LSTM's weights (PyTorch's default
            # U(-1/sqrt(H), 1/sqrt(H)) init) and the loss gradient at the last
            # hidden state; the forward pass gives what it stores
            rE = _rng(wl.wid, tid); tid += 1
            rW = _rng(wl.wid, tid); tid += 1
            rD = _rng(wl.wid, tid); tid += 1
            emb = by_name_emb(wl)
            E = _normal(rE, (emb.V, emb.D))
            k = 1.0 / np.sqrt(layer.H)
            G = 4 * layer.H
            W_ih = rW.uniform(-k, k, (G, layer.D)).astype(np.float32)
            W_hh = rW.uniform(-k, k, (G, layer.H)).astype(np.float32)
            b_ih = rW.uniform(-k, k, G).astype(np.float32)
            b_hh = rW.uniform(-k, k, G).astype(np.float32)
            x = E[emb_ids].astype(np.float32)
            gates, c, h = lstm_forward_activations(x.astype(np.float64), W_ih.astype(np.float64),
                                                   W_hh.astype(np.float64), b_ih.astype(np.float64),
                                                   b_hh.astype(np.float64))
            lstm_fwd = (x, h.astype(np.float32))
            li.aux = {"gates": gates.astype(np.float32), "c": c.astype(np.float32), "W_hh": W_hh,
                      "dh_last": _normal(rD, (N, layer.H)) / np.float32(wl.N)}
        elif isinstance(layer, LayerNorm):
            rA = _rng(wl.wid, tid); tid += 1
            rB = _rng(wl.wid, tid); tid += 1
            li.A = _normal(rA, (N, layer.T, layer.D))
            li.B = _normal(rB, (N, layer.T, layer.D)) / np.float32(wl.N)
        elif isinstance(layer, GroupNorm):
            # A: the normalized input xhat [N, C, P]
            rA = _rng(wl.wid, tid); tid += 1
            rB = _rng(wl.wid, tid); tid += 1
            li.A = _normal(rA, (N, layer.C, layer.P))
            li.B = _normal(rB, (N, layer.C, layer.P)) / np.float32(wl.N)
        else:
            raise TypeError(layer)
        out.append(li)
        by_name[layer.name] = li
    return out


# entries of LayerInputs.aux that are per sample (the first axis is the batch)
_AUX_PER_SAMPLE = ("gates", "c", "dh_last")


def take_samples(inputs: List[LayerInputs], idx) -> List[LayerInputs]:
    """The same layers' inputs for the samples ``idx`` (an index array or a slice)."""
    out = []
    for li in inputs:
        aux = None
        if li.aux is not None:
            aux = {k: (v[idx] if k in _AUX_PER_SAMPLE else v) for k, v in li.aux.items()}
        out.append(LayerInputs(li.layer, A=None if li.A is None else li.A[idx],
                               B=None if li.B is None else li.B[idx],
                               ids=None if li.ids is None else li.ids[idx], aux=aux))
    return out


def by_name_emb(wl: Workload) -> Embedding:
    for l in wl.layers:
        if isinstance(l, Embedding):
            return l
    raise ValueError("workload has no embedding")


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest-even) and return the raw uint16 bits."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to fp32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def rounded_like_device(wl: Workload, a: Optional[np.ndarray]) -> Optional[np.ndarray]:
    """The values the device consumes, widened to fp32 (identity for fp32 workloads)."""
    if a is None or wl.dtype == F32:
        return a
    return bf16_bits_to_f32(to_bf16_bits(a))
