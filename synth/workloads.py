"""Workload shapes and seeded random inputs (no optimizer arithmetic here)."""
import math
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Shapes
# ---------------------------------------------------------------------------

VOCAB = 30522
POSITIONS = 512


def bert_tensor_shapes(layers: int, hidden: int, ffn: int) -> List[Tuple[Tuple[int, ...], int]]:
    """BERT encoder tensors as ((shape), fan_in), in order: word embedding,
    position embedding, then per layer Q, K, V, O weights and biases, FFN in
    (weight, bias), FFN out (weight, bias), and two LayerNorms (gamma, beta).
    2-D weights are [out, in]; fan_in is the column count (embeddings: the
    hidden size).  1-D tensors get fan_in 1 (gradient scale 1)."""
    t = [((VOCAB, hidden), hidden), ((POSITIONS, hidden), hidden)]
    for _ in range(layers):
        for _qkvo in range(4):
            t.append(((hidden, hidden), hidden))
            t.append(((hidden,), 1))
        t.append(((ffn, hidden), hidden))
        t.append(((ffn,), 1))
        t.append(((hidden, ffn), ffn))
        t.append(((hidden,), 1))
        for _ln in range(2):
            t.append(((hidden,), 1))
            t.append(((hidden,), 1))
    return t


def stress_sizes(count: int = 5000, lo: int = 64, hi: int = 1 << 20, seed: int = 2) -> List[int]:
    """Tensor sizes log-uniform in [lo, hi], seeded."""
    rng = np.random.Generator(np.random.Philox(key=[seed, 0x5157]))
    u = rng.uniform(math.log(lo), math.log(hi), size=count)
    return [int(min(hi, max(lo, round(math.exp(a))))) for a in u]


@dataclass
class Workload:
    name: str
    numel: List[int]                 # compressed tensors (each chunked into n)
    n: int                           # workers
    warmup_steps: int
    steps: int
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    param_std: float = 0.02
    grad_std: float = 1e-3
    # gradient scale per range of the flat buffer: list of (numel, scale)
    grad_scale_ranges: Optional[List[Tuple[int, float]]] = None
    n_local: Optional[int] = None    # workers simulated on this GPU (default n)
    server_chunk: Optional[int] = None  # real-share: the one chunk this GPU serves
    seed_params: int = 0
    seed_grads: int = 1
    seed_incoming: int = 3
    description: str = ""

    @property
    def d(self) -> int:
        return int(sum(self.numel))

    @property
    def local_workers(self) -> int:
        return self.n if self.n_local is None else self.n_local


def _bert(name, layers, hidden, n, warmup, steps, desc):
    shapes = bert_tensor_shapes(layers, hidden, 4 * hidden)
    ranges = [(int(np.prod(s)), 1.0 / math.sqrt(f)) for s, f in shapes]
    d = sum(r[0] for r in ranges)
    return Workload(name=name, numel=[d], n=n, warmup_steps=warmup, steps=steps,
                    grad_scale_ranges=ranges, description=desc)


def _make_workloads():
    w = {}
    w["tiny"] = Workload(
        name="tiny", numel=[1 << 20], n=4, warmup_steps=10, steps=10,
        description="one flat fp32 tensor d=2^20, n=4 simulated workers")
    w["bert_base"] = _bert(
        "bert_base", 12, 768, 16, 5, 20,
        "BERT-Base-shaped flat fp32 buffer (194 tensors, d=108,888,576), n=16")
    w["bert_large"] = _bert(
        "bert_large", 24, 1024, 32, 5, 20,
        "BERT-Large-shaped flat fp32 buffer (386 tensors, d=334,088,192), n=32")
    w["stress"] = Workload(
        name="stress", numel=stress_sizes(), n=8, warmup_steps=5, steps=10,
        description="5,000 fp32 tensors, log-uniform sizes in [64, 2^20], "
                    "compressed per tensor, n=8")
    share = _bert("share256", 24, 1024, 256, 5, 1,
                  "one GPU's share of a 256-worker BERT-Large step: one local "
                  "worker over d, server of chunk 0 from 256 incoming chunks")
    share.n_local = 1
    share.server_chunk = 0
    w["share256"] = share
    return w


WORKLOADS = _make_workloads()


def get(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------------------
# Host (numpy) generators
# ---------------------------------------------------------------------------

def _rng(seed: int, a: int = 0, b: int = 0) -> np.random.Generator:
    key = np.array([(seed << 40) ^ a, b], dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def host_normal(size, std, seed, a=0, b=0) -> np.ndarray:
    return (_rng(seed, a, b).standard_normal(size, dtype=np.float32)
            * np.float32(std)).astype(np.float32)


def grad_scale_per_element(wl: Workload, D: int, tensor_off) -> np.ndarray:
    """Per-element gradient standard deviation over the padded buffer."""
    s = np.zeros(D, np.float32)
    if wl.grad_scale_ranges is None:
        for off, d in zip(tensor_off, wl.numel):
            s[off:off + d] = wl.grad_std
    else:
        assert len(wl.numel) == 1
        pos = int(tensor_off[0])
        for cnt, sc in wl.grad_scale_ranges:
            s[pos:pos + cnt] = np.float32(wl.grad_std * sc)
            pos += cnt
    return s


def host_params(wl: Workload, D: int) -> np.ndarray:
    return host_normal(D, wl.param_std, wl.seed_params)


def host_grads(wl: Workload, D: int, tensor_off, step: int, workers=None) -> np.ndarray:
    """[len(workers), D] gradients for one step; padding elements are 0."""
    workers = list(range(wl.local_workers)) if workers is None else list(workers)
    scale = grad_scale_per_element(wl, D, tensor_off)
    out = np.empty((len(workers), D), np.float32)
    for r, i in enumerate(workers):
        out[r] = _rng(wl.seed_grads, step, i).standard_normal(D, dtype=np.float32) * scale
    return out


def host_bits_and_scales(rows: int, words: int, seed: int, mu=-7.0, sigma=0.5):
    """Incoming packed sign words (Bernoulli(0.5) bits) and lognormal scales."""
    rng = _rng(seed, 0x1B17, 0)
    bits = rng.integers(0, np.iinfo(np.uint64).max, size=(rows, words),
                        dtype=np.uint64, endpoint=True)
    scales = np.exp(rng.normal(mu, sigma, size=rows)).astype(np.float32)
    return bits, scales


# ---------------------------------------------------------------------------
# Device (torch) generators -- for the full-size workloads
# ---------------------------------------------------------------------------

def _gen(device, seed: int, a: int = 0, b: int = 0):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(((seed * 1000003 + a) * 1000003 + b) & ((1 << 62) - 1))
    return g


def device_params(wl: Workload, D: int, device):
    import torch
    x = torch.empty(D, dtype=torch.float32, device=device)
    x.normal_(0.0, wl.param_std, generator=_gen(device, wl.seed_params))
    return x


def device_grads(wl: Workload, D: int, tensor_off, step: int, out, scale_vec=None):
    """Fills out[rows, >=D] with one step's gradients of workers 0..rows-1.
    scale_vec: optional per-element std (device tensor [D])."""
    import torch
    if scale_vec is None:
        scale_vec = torch.from_numpy(grad_scale_per_element(wl, D, tensor_off)).to(out.device)
    for i in range(out.shape[0]):
        row = out[i, :D]
        row.normal_(0.0, 1.0, generator=_gen(out.device, wl.seed_grads, step, i))
        row.mul_(scale_vec)
    return out


def device_bits_and_scales(rows: int, words: int, seed: int, device, mu=-7.0, sigma=0.5):
    import torch
    g = _gen(device, seed, 0x1B17)
    raw = torch.randint(-(1 << 31), 1 << 31, (rows, 2 * words), dtype=torch.int32,
                        device=device, generator=g)
    bits = raw.view(torch.int64)
    scales = torch.empty(rows, dtype=torch.float32, device=device)
    scales.log_normal_(mu, sigma, generator=g)
    return bits, scales
