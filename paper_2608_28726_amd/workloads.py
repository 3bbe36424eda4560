"""Seeded synthetic inputs shaped like the verifier's workloads.

The paper measures on its benchmark suite with three small multimodal
models (Sec. 4.1); neither data nor weights are available, so these seeded
generators stand in for the logit rows those models emit. This module draws
inputs only: it computes none of the verifier's features, and both the HIP
path and the oracle read the logits it stores.

Row model (every configuration): z_v = s_r * g_v with g_v ~ N(0, 1) i.i.d.,
plus a spike of height h_r on one token j_r ~ U{0..V-1}; generated in
float32 and rounded to bfloat16 (round-to-nearest-even) for bf16 workloads.

The logits come from a counter-based generator with two implementations
that produce the same bits: numpy on the host (:func:`host_rows`) and a HIP
kernel on the device (``libprtools.so``, csrc/tools/prtools.hip). Element v
of row r is a pure function of (seed, r, v): 64 bits from the SplitMix64
output function (Steele, Lea and Flood, OOPSLA 2014) on a Weyl sequence,
turned into a normal deviate by a piecewise-linear quantile table (cells of
2^-16 of probability, the two outermost refined to cells of 2^-32), then
scaled by s_r in float32. Because both sides agree bit for bit, expected
values can be computed on a host from host-made rows and compared with GPU
outputs on device-made rows; :func:`row_checksums` confirms the agreement.

The sampled token is drawn from softmax(z / T) by the Gumbel-max trick; with
top-p on it is drawn by inverse CDF at u * P over the tokens sorted by
logit, which always lands inside the nucleus (the engine's top-p sampler,
an input recipe rather than part of the verifier). Host-made batches draw it
in float64 numpy from counter-based uniforms; device-made batches draw it
with torch on the device (same distribution, other draws) unless the caller
passes the ids.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from statistics import NormalDist

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

# The 512 x 512 offline workload is processed as this many chunks of whole
# requests, chunk c being workload ``scaled(w, n_req=512 // 16, seed=w.seed + c)``.
OFFLINE_CHUNKS = 16


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


def offline_chunk(w: Workload, c: int) -> Workload:
    """Chunk c of the offline workload (whole requests, its own seed)."""
    return scaled(w, n_req=w.n_req // OFFLINE_CHUNKS, seed=w.seed + c)


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


# ---------------------------------------------------------------------------
# The counter-based logit generator (host twin of csrc/tools/prtools.hip)

_MASK64 = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB
_IDS_SALT = 0x5A5A5A5A5A5A5A5A  # key of the host sampler's uniforms
_STREAM_SALT = 0x53545245414D0000  # key of the streaming workload's rows


def mix64_int(x: int) -> int:
    """SplitMix64's output function on one 64-bit integer."""
    x &= _MASK64
    x = ((x ^ (x >> 30)) * _MIX1) & _MASK64
    x = ((x ^ (x >> 27)) * _MIX2) & _MASK64
    return x ^ (x >> 31)


def mix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64's output function, element-wise on uint64 (wrapping)."""
    x = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        x = (x ^ (x >> np.uint64(30))) * np.uint64(_MIX1)
        x = (x ^ (x >> np.uint64(27))) * np.uint64(_MIX2)
    return x ^ (x >> np.uint64(31))


def row_key(seed: int, r: int) -> int:
    return mix64_int((seed & _MASK64) + ((r + 1) * _GAMMA & _MASK64))


_WEYL_CACHE: dict = {}


def _weyl(V: int) -> np.ndarray:
    """(v + 1) * G mod 2^64 for v < V."""
    t = _WEYL_CACHE.get(V)
    if t is None:
        with np.errstate(over="ignore"):
            t = (np.arange(V, dtype=np.uint64) + np.uint64(1)) * np.uint64(_GAMMA)
        _WEYL_CACHE.clear()
        _WEYL_CACHE[V] = t
    return t


def element_bits(key: int, V: int) -> np.ndarray:
    """The 64 random bits of each element of a row with this key."""
    with np.errstate(over="ignore"):
        return mix64(np.uint64(key) + _weyl(V))


_TABLES = None


def normal_tables():
    """The quantile tables (A_i, D_i) as float32 [65536, 2] arrays (main, tail).

    main: A_i = Q(i / 2^16) for 1 <= i <= 65535, D_i = A_{i+1} - A_i
    (cells 0 and 65535 are not read). tail: A_j = Q(j / 2^32) for
    1 <= j <= 65536, A_0 = Q(2^-34) standing in for -inf, D_j = A_{j+1} - A_j.
    Q is the standard normal quantile function in float64 (Python's
    statistics.NormalDist), rounded to float32; the differences are float32.
    """
    global _TABLES
    if _TABLES is None:
        Q = NormalDist().inv_cdf
        A = np.zeros(65537, dtype=np.float32)
        A[1:65536] = np.array([Q(i / 65536.0) for i in range(1, 65536)], dtype=np.float64).astype(np.float32)
        main = np.zeros((65536, 2), dtype=np.float32)
        main[:, 0] = A[:65536]
        main[1:65535, 1] = A[2:65536] - A[1:65535]
        At = np.empty(65537, dtype=np.float32)
        At[0] = np.float32(Q(2.0 ** -34))
        At[1:] = np.array([Q(j * 2.0 ** -32) for j in range(1, 65537)], dtype=np.float64).astype(np.float32)
        tail = np.empty((65536, 2), dtype=np.float32)
        tail[:, 0] = At[:65536]
        tail[:, 1] = At[1:] - At[:65536]
        _TABLES = (main, tail)
    return _TABLES


def normal_from_bits(b: np.ndarray) -> np.ndarray:
    """float32 normal deviates from 64-bit words (see the module docstring)."""
    main, tail = normal_tables()
    hi = (b >> np.uint64(32)).astype(np.uint32)
    cell = hi >> np.uint32(16)
    frac = (hi & np.uint32(0xFFFF)).astype(np.float32) * np.float32(1.0 / 65536.0)
    t = main[cell]
    g = t[:, 0] + frac * t[:, 1]
    out = np.flatnonzero((cell == 0) | (cell == 65535))
    if out.size:
        lo = b[out].astype(np.uint32)  # the low 32 bits
        tt = tail[lo >> np.uint32(16)]
        gt = tt[:, 0] + ((lo & np.uint32(0xFFFF)).astype(np.float32) * np.float32(1.0 / 65536.0)) * tt[:, 1]
        g[out] = np.where(cell[out] == 0, gt, -gt)
    return g


def bf16_bits(z: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16, as uint16 bit patterns (finite inputs)."""
    b = np.asarray(z, dtype=np.float32).view(np.uint32)
    return ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def host_row(seed: int, r: int, V: int, dtype: str, s: float, h: float, j: int) -> np.ndarray:
    """One generated row on the host: float32 values, or bf16 bits as uint16."""
    z = np.float32(s) * normal_from_bits(element_bits(row_key(seed, r), V))
    if 0 <= j < V:
        z[j] = z[j] + np.float32(h)
    return bf16_bits(z) if dtype == "bf16" else z


def host_rows(seed: int, row_index, V: int, dtype: str, s, h, j) -> np.ndarray:
    """Generated rows [len(row_index), V] on the host (float32, or bf16 bits as uint16)."""
    row_index = np.asarray(row_index, dtype=np.int64)
    out = np.empty((row_index.shape[0], V), dtype=np.uint16 if dtype == "bf16" else np.float32)
    for k, r in enumerate(row_index):
        out[k] = host_row(seed, int(r), V, dtype, float(s[k]), float(h[k]), int(j[k]))
    return out


_TOOLS = None
_DEV_TABLES: dict = {}


def tools():
    """libprtools.so (built beside libprouter.so). Raises ImportError when missing."""
    global _TOOLS
    if _TOOLS is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libprtools.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with `python -m paper_2608_28726_amd.build`")
        L = ctypes.CDLL(path)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.prt_fill_logits.argtypes = [vp, ctypes.c_int, i64, i32, i64, ctypes.c_uint64, i64, vp, vp, vp, vp, vp,
                                      vp, vp]
        L.prt_fill_logits.restype = ctypes.c_int
        L.prt_read_probe.argtypes = [vp, i64, vp, i32, i32, i32, vp]
        L.prt_read_probe.restype = ctypes.c_int
        L.prt_exp2_max_rel_err.argtypes = [ctypes.c_float, ctypes.c_float, vp, vp]
        L.prt_exp2_max_rel_err.restype = ctypes.c_int
        _TOOLS = L
    return _TOOLS


def _device_tables(dev):
    key = str(dev)
    if key not in _DEV_TABLES:
        main, tail = normal_tables()
        _DEV_TABLES[key] = (torch.from_numpy(main).to(dev), torch.from_numpy(tail).to(dev))
    return _DEV_TABLES[key]


def fill_logits(out: torch.Tensor, s: np.ndarray, h: np.ndarray, j: np.ndarray, seed: int, row0: int = 0,
                row_index: np.ndarray | None = None) -> torch.Tensor:
    """Fills out[n_rows, V] (float32 or bfloat16) with generated rows r0 ..
    (key index row_index[k], or row0 + k) on out's device."""
    n, V = out.shape
    dev = out.device
    idx = np.arange(row0, row0 + n, dtype=np.int64) if row_index is None else np.asarray(row_index, np.int64)
    dtype = "bf16" if out.dtype == torch.bfloat16 else "f32"
    if dev.type == "cpu":
        raw = host_rows(seed, idx, V, dtype, s, h, j)
        src = torch.from_numpy(raw.view(np.int16)).view(torch.bfloat16) if dtype == "bf16" else torch.from_numpy(raw)
        out.copy_(src)
        return out
    main, tail = _device_tables(dev)
    args = [torch.as_tensor(np.asarray(a), device=dev) for a in
            (idx, np.asarray(s, np.float32), np.asarray(h, np.float32), np.asarray(j, np.int64))]
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    st = tools().prt_fill_logits(ctypes.c_void_p(out.data_ptr()), 1 if dtype == "bf16" else 0, n, V, out.stride(0),
                                 ctypes.c_uint64(seed & _MASK64), 0, ctypes.c_void_p(args[0].data_ptr()),
                                 *(ctypes.c_void_p(a.data_ptr()) for a in args[1:]),
                                 ctypes.c_void_p(main.data_ptr()), ctypes.c_void_p(tail.data_ptr()), stream)
    if st != 0:
        raise RuntimeError(f"prt_fill_logits failed with status {st}")
    return out  # the argument tensors are freed in stream order, after the kernel


# ---------------------------------------------------------------------------
# Checksums of stored rows (host and device agree on the bits)

CHECKSUM_MOD = (1 << 61) - 1


def row_checksums(x, chunk_rows: int = 256) -> np.ndarray:
    """Per-row checksum of stored logits: sum_v c_v * ((v mod 65521) + 1), with
    c_v the 16-bit pattern of a bf16 logit, or lo16 + 7 hi16 of a float32's
    bits. ``x`` is a torch tensor (any device) or a numpy raw array
    (float32 values or bf16 bits as uint16). Returns int64[n_rows]."""
    if isinstance(x, np.ndarray):
        x = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16) if x.dtype == np.uint16 else torch.from_numpy(x)
    n, V = x.shape
    dev = x.device
    w = torch.arange(V, device=dev, dtype=torch.int64) % 65521 + 1
    out = torch.empty(n, dtype=torch.int64, device=dev)
    for r0 in range(0, n, chunk_rows):
        blk = x[r0:r0 + chunk_rows]
        if blk.dtype == torch.bfloat16:
            c = (blk.view(torch.int16).to(torch.int64) & 0xFFFF) * w
            out[r0:r0 + chunk_rows] = c.sum(1)
        else:
            bits = blk.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
            out[r0:r0 + chunk_rows] = ((bits & 0xFFFF) * w).sum(1) + 7 * ((bits >> 16) * w).sum(1)
    return out.cpu().numpy()


def combine_checksums(c) -> int:
    """One checksum of a group of rows, in order: sum_k c_k (k + 1) mod 2^61 - 1."""
    return sum(int(v) * (k + 1) for k, v in enumerate(np.asarray(c).tolist())) % CHECKSUM_MOD


# ---------------------------------------------------------------------------
# Batches

def request_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(w.len_lo, w.len_hi + 1, size=w.n_req).astype(np.int64)


def row_params(w: Workload, n_rows: int, rng: np.random.Generator):
    s = rng.uniform(w.s_lo, w.s_hi, size=n_rows).astype(np.float32)
    h = rng.uniform(w.h_lo, w.h_hi, size=n_rows).astype(np.float32)
    j = rng.integers(0, w.V, size=n_rows).astype(np.int64)
    return s, h, j


def _decode(raw_row: np.ndarray) -> np.ndarray:
    if raw_row.dtype == np.uint16:
        return (raw_row.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return raw_row.astype(np.float64)


def host_sample_ids(raw: np.ndarray, temperature, top_p, seed: int, row_index) -> np.ndarray:
    """Sampled token of each host row (see the module docstring), float64.
    Uniforms come from the counter-based bits keyed on (seed ^ salt, row index)."""
    n, V = raw.shape
    out = np.empty(n, dtype=np.int32)
    idx = np.arange(V)
    for k in range(n):
        key = row_key(seed ^ _IDS_SALT, int(row_index[k]))
        z = _decode(raw[k])
        T = float(np.float32(temperature[k]))
        P = None if top_p is None else float(np.float32(top_p[k]))
        if P is None or P >= 1.0:
            b = element_bits(key, V)
            u = ((b >> np.uint64(11)).astype(np.float64) + 0.5) * 2.0 ** -53
            with np.errstate(divide="ignore"):
                g = -np.log(-np.log(u))
            out[k] = int(np.argmax(z / T + g))
        else:
            order = np.lexsort((idx, -z))
            zs = z[order]
            wgt = np.exp((zs - zs[0]) / T)
            cdf = np.cumsum(wgt)
            u = ((mix64_int(key) >> 11) + 0.5) * 2.0 ** -53
            pos = min(int(np.searchsorted(cdf, u * P * cdf[-1])), V - 1)
            out[k] = int(order[pos])
    return out


def sample_ids(logits: torch.Tensor, temperature: torch.Tensor, top_p: torch.Tensor | None, seed: int,
               chunk_rows: int = 256) -> torch.Tensor:
    """Sampled token per row of device-made logits, drawn with torch on the
    logits' device (see the module docstring)."""
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


def batch_plan(w: Workload, lengths: np.ndarray | None = None):
    """Offsets and per-row parameters of workload w's batch (host numpy):
    offsets, s, h, j, T per row, P per row (or None)."""
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
    return offsets, s, h, j, T_row, P_row


def make_batch(w: Workload, device="cpu", lengths: np.ndarray | None = None, ids=None) -> Batch:
    """A seeded offline batch of workload `w` (logits generated on `device`).
    ``ids`` (int32 per row) replaces the drawn sampled tokens."""
    offsets, s, h, j, T_row, P_row = batch_plan(w, lengths)
    n = int(offsets[-1])
    logits = torch.empty((n, w.V), dtype=w.torch_dtype, device=device)
    fill_logits(logits, s, h, j, seed=w.seed)
    temperature = torch.as_tensor(T_row, device=device)
    top_p = None if P_row is None else torch.as_tensor(P_row, device=device)
    if ids is not None:
        ids = torch.as_tensor(np.asarray(ids, dtype=np.int32), device=device)
    elif torch.device(device).type == "cpu":
        ids = torch.from_numpy(host_sample_ids(to_host_raw(logits), T_row, P_row, w.seed, np.arange(n)))
    else:
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


def stream_rows(w: Workload, step: int, active: np.ndarray):
    """Key indices and row parameters of the active slots' rows at a decode
    step: each (step, slot) row is a function of the pair alone."""
    active = np.asarray(active, dtype=np.int64)
    rng = np.random.default_rng([w.seed, step])
    s, h, j = row_params(w, w.n_req, rng)
    return (step - 1) * w.n_req + active, s[active], h[active], j[active]


def stream_seed(w: Workload) -> int:
    return w.seed ^ _STREAM_SALT


def stream_step_inputs(w: Workload, step: int, active: np.ndarray, device="cpu", ids=None):
    """Logits, ids and temperatures of one decode step for the `active` slots."""
    n = len(active)
    idx, s, h, j = stream_rows(w, step, active)
    logits = torch.empty((n, w.V), dtype=w.torch_dtype, device=device)
    fill_logits(logits, s, h, j, seed=stream_seed(w), row_index=idx)
    T_row = np.full(n, np.float32(w.T_lo), dtype=np.float32)
    T = torch.as_tensor(T_row, device=device)
    if ids is not None:
        ids = torch.as_tensor(np.asarray(ids, dtype=np.int32), device=device)
    elif torch.device(device).type == "cpu":
        ids = torch.from_numpy(host_sample_ids(to_host_raw(logits), T_row, None, stream_seed(w), idx))
    else:
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
