"""Seeded synthetic inputs shaped like the verifier's workloads.

The paper measures on its benchmark suite with three small multimodal
models (Sec. 4.1); neither data nor weights are available, so these seeded
generators stand in for the logit rows those models emit. This module draws
inputs only: it computes none of the verifier's features, and both the HIP
path and the oracle read the logits it stores.

Row model (every configuration): z_v = s_r * g_v with g_v ~ N(0, 1) i.i.d.,
plus a spike of height h_r on one token j_r ~ U{0..V-1}; generated in
float32 and rounded to bfloat16 (round-to-nearest-even) for bf16 workloads.
The sampled token is drawn from softmax(z / T) by the Gumbel-max trick; with
top-p on it is drawn by inverse CDF at u * P over the tokens sorted by
logit, which always lands inside the nucleus (the engine's top-p sampler,
an input recipe rather than part of the verifier).
"""

from __future__ import annotations

import dataclasses

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    n_req: int
    len_lo: int  # request lengths ~ U{len_lo..len_hi}
    len_hi: int
    V: int
    dtype: str  # "f32" | "bf16"
    s_lo: float
    s_hi: float
    h_lo: float
    h_hi: float
    T_lo: float  # per-request temperature ~ U[T_lo, T_hi] (equal: fixed)
    T_hi: float
    P_lo: float | None = None  # per-request top-p ~ U[P_lo, P_hi]; None: off
    P_hi: float | None = None
    tau: float = 0.5
    q: float = 0.1
    seed: int = 0

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


WORKLOADS = {
    "pr1_ref_8x64_v32000_f32": Workload(
        "pr1_ref_8x64_v32000_f32", "8 requests x 64 tokens, V=32,000 float32, T=1, no top-p",
        8, 64, 64, 32000, "f32", 1.0, 4.0, 0.0, 15.0, 1.0, 1.0, seed=0x50520001),
    "ragged_64req_v151936_bf16": Workload(
        "ragged_64req_v151936_bf16", "64 requests, lengths U{16..512}, V=151,936 bfloat16, T=0.7, no top-p",
        64, 16, 512, 151936, "bf16", 1.0, 4.0, 0.0, 15.0, 0.7, 0.7, seed=0x50520002),
    "stream_256slots_v151936_bf16": Workload(
        "stream_256slots_v151936_bf16",
        "256 concurrent requests finishing at step U{32..1024}, one V=151,936 bfloat16 row each per step, T=1",
        256, 32, 1024, 151936, "bf16", 1.0, 4.0, 0.0, 15.0, 1.0, 1.0, seed=0x50520003),
    "offline_512x512_v151936_bf16": Workload(
        "offline_512x512_v151936_bf16", "512 requests x 512 tokens, V=151,936 bfloat16, s~U[0.5,5], h~U[0,20], T=1",
        512, 512, 512, 151936, "bf16", 0.5, 5.0, 0.0, 20.0, 1.0, 1.0, seed=0x50520004),
    "topp_128x256_v262144_f32": Workload(
        "topp_128x256_v262144_f32",
        "128 requests x 256 tokens, V=262,144 float32, T~U[0.3,1.2], top-p~U[0.8,0.95] per request",
        128, 256, 256, 262144, "f32", 1.0, 4.0, 0.0, 15.0, 0.3, 1.2, 0.8, 0.95, seed=0x50520005),
}


def scaled(w: Workload, n_req: int | None = None, len_hi: int | None = None, V: int | None = None,
           **kw) -> Workload:
    """The same row model at a smaller shape (parity tests)."""
    changes = {}
    if n_req is not None:
        changes["n_req"] = n_req
    if len_hi is not None:
        changes["len_hi"] = len_hi
        changes["len_lo"] = min(w.len_lo, len_hi)
    if V is not None:
        changes["V"] = V
    changes.update(kw)
    return dataclasses.replace(w, **changes)


@dataclasses.dataclass
class Batch:
    """One offline batch: logits [n_rows, V] plus per-row inputs, on `device`."""
    workload: Workload
    offsets: np.ndarray  # int32 [n_req + 1]
    logits: torch.Tensor
    sampled_ids: torch.Tensor  # int32 [n_rows]
    temperature: torch.Tensor  # float32 [n_rows]
    top_p: torch.Tensor | None  # float32 [n_rows]

    @property
    def n_rows(self) -> int:
        return int(self.offsets[-1])


def request_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(w.len_lo, w.len_hi + 1, size=w.n_req).astype(np.int64)


def row_params(w: Workload, n_rows: int, rng: np.random.Generator):
    s = rng.uniform(w.s_lo, w.s_hi, size=n_rows).astype(np.float32)
    h = rng.uniform(w.h_lo, w.h_hi, size=n_rows).astype(np.float32)
    j = rng.integers(0, w.V, size=n_rows).astype(np.int64)
    return s, h, j


def fill_logits(out: torch.Tensor, s: np.ndarray, h: np.ndarray, j: np.ndarray, seed: int,
                chunk_rows: int = 1024) -> torch.Tensor:
    """Fills out[n_rows, V] (float32 or bfloat16) with the spike-plus-Gaussian rows."""
    n, V = out.shape
    dev = out.device
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        z = torch.randn((r1 - r0, V), generator=gen, device=dev, dtype=torch.float32)
        z.mul_(torch.as_tensor(s[r0:r1], device=dev).unsqueeze(1))
        rows = torch.arange(r1 - r0, device=dev)
        cols = torch.as_tensor(j[r0:r1], device=dev)
        z[rows, cols] += torch.as_tensor(h[r0:r1], device=dev)
        out[r0:r1].copy_(z)  # float32 -> bfloat16 rounds to nearest even
    return out


def sample_ids(logits: torch.Tensor, temperature: torch.Tensor, top_p: torch.Tensor | None, seed: int,
               chunk_rows: int = 256) -> torch.Tensor:
    """Sampled token per row (see the module docstring)."""
    n, V = logits.shape
    dev = logits.device
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed ^ 0x5A5A5A5A)
    out = torch.empty(n, dtype=torch.int32, device=dev)
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        u = logits[r0:r1].float() / temperature[r0:r1].unsqueeze(1)
        if top_p is None:
            g = torch.rand((r1 - r0, V), generator=gen, device=dev, dtype=torch.float32)
            g.clamp_(min=1e-38).log_().neg_().log_().neg_()  # Gumbel(0, 1)
            out[r0:r1] = torch.argmax(u + g, dim=1).to(torch.int32)
        else:
            vals, idx = torch.sort(u.double(), dim=1, descending=True)
            w = torch.exp(vals - vals[:, :1])
            cdf = torch.cumsum(w, dim=1)
            P = top_p[r0:r1].double().clamp(max=1.0)
            ur = torch.rand(r1 - r0, generator=gen, device=dev, dtype=torch.float64)
            target = (ur * P * cdf[:, -1]).unsqueeze(1)
            pos = torch.searchsorted(cdf, target).clamp(max=V - 1)
            out[r0:r1] = idx.gather(1, pos).squeeze(1).to(torch.int32)
    return out


def make_batch(w: Workload, device="cpu", lengths: np.ndarray | None = None) -> Batch:
    """A seeded offline batch of workload `w` (logits generated on `device`)."""
    rng = np.random.default_rng(w.seed)
    if lengths is None:
        lengths = request_lengths(w, rng)
    offsets = np.zeros(len(lengths) + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lengths)
    n = int(offsets[-1])
    s, h, j = row_params(w, n, rng)
    T_req = rng.uniform(w.T_lo, w.T_hi, size=len(lengths)).astype(np.float32)
    T_row = np.repeat(T_req, lengths)
    P_row = None
    if w.P_lo is not None:
        P_req = rng.uniform(w.P_lo, w.P_hi, size=len(lengths)).astype(np.float32)
        P_row = np.repeat(P_req, lengths)
    logits = torch.empty((n, w.V), dtype=w.torch_dtype, device=device)
    fill_logits(logits, s, h, j, seed=w.seed)
    temperature = torch.as_tensor(T_row, device=device)
    top_p = None if P_row is None else torch.as_tensor(P_row, device=device)
    ids = sample_ids(logits, temperature, top_p, seed=w.seed)
    return Batch(w, offsets, logits, ids, temperature, top_p)


def stream_schedule(w: Workload, n_steps: int | None = None) -> np.ndarray:
    """Finish step f_i ~ U{len_lo..len_hi} of each of the w.n_req slots (all
    start at step 1; no refill). Step s (1-based) has the slots with f_i >= s."""
    rng = np.random.default_rng(w.seed)
    f = rng.integers(w.len_lo, w.len_hi + 1, size=w.n_req).astype(np.int64)
    if n_steps is not None:
        f = np.minimum(f, n_steps)
    return f


def stream_step_inputs(w: Workload, step: int, active: np.ndarray, device="cpu"):
    """Logits, ids and temperatures of one decode step for the `active` slots."""
    n = len(active)
    rng = np.random.default_rng([w.seed, step])
    s, h, j = row_params(w, n, rng)
    logits = torch.empty((n, w.V), dtype=w.torch_dtype, device=device)
    fill_logits(logits, s, h, j, seed=(w.seed * 1_000_003 + step) & 0x7FFFFFFFFFFF)
    T = torch.full((n,), float(np.float32(w.T_lo)), dtype=torch.float32, device=device)
    ids = sample_ids(logits, T, None, seed=(w.seed + step) & 0x7FFFFFFF)
    return logits, ids, T


def to_host_raw(logits: torch.Tensor) -> np.ndarray:
    """The stored logits as numpy: float32 values, or bfloat16 bit patterns as uint16."""
    t = logits.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


# Parameter tensors of the verifier head in storage order, with the fan-in
# that scales their synthetic initial values (input recipe only; the layout
# itself is documented with pr_verifier_head in include/prouter.h).
_HEAD_TENSORS = (
    [("W_in", 64 * 4, 4), ("b_in", 64, 4)]
    + [t for _ in range(2) for t in (
        ("W_qkv", 192 * 64, 64), ("b_qkv", 192, 64), ("W_o", 64 * 64, 64), ("b_o", 64, 64),
        ("ln1_g", 64, None), ("ln1_b", 64, None), ("W_1", 128 * 64, 64), ("b_1", 128, 64),
        ("W_2", 64 * 128, 128), ("b_2", 64, 128), ("ln2_g", 64, None), ("ln2_b", 64, None))]
    + [("w_out", 64, 64), ("b_out", 1, 64)]
)


def head_weights(seed: int = 0x50524844) -> np.ndarray:
    """Seeded synthetic weights of the verifier head (the paper publishes
    none): linear weights and biases ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in)),
    LayerNorm gains ~ 1 + U(-0.1, 0.1) and shifts ~ U(-0.1, 0.1). Flat
    float32, 67,329 entries."""
    rng = np.random.default_rng(seed)
    parts = []
    for name, n, fan_in in _HEAD_TENSORS:
        if fan_in is None:
            v = rng.uniform(-0.1, 0.1, n) + (1.0 if name.endswith("_g") else 0.0)
        else:
            a = 1.0 / np.sqrt(fan_in)
            v = rng.uniform(-a, a, n)
        parts.append(v.astype(np.float32))
    return np.concatenate(parts)


def validation_scores(n: int, seed: int = 0x50524341, nan_frac: float = 0.005) -> np.ndarray:
    """A seeded validation pool of n shipping confidences in (0, 1), skewed
    towards confident requests (Beta(5, 2)), with a fraction of NaN (requests
    without a score). float32."""
    rng = np.random.default_rng(seed)
    s = rng.beta(5.0, 2.0, n).astype(np.float32)
    s[rng.random(n) < nan_frac] = np.nan
    return s
