"""Token-aware verifier hot path on MI355X (Pro-Router, Sec. 3.1).

A thin binding over the C ABI of ``libprouter.so`` (include/prouter.h):
tensors are checked and their device pointers handed to the library, which
runs every step of the path in its own HIP kernels on torch's current
stream. PyTorch only provides device memory and streams here.

    feats = token_features(logits, sampled_ids, temperature, top_p=None)
    agg = request_aggregate(feats, offsets)
    ship, n_ship = route(agg["score"], threshold)

The paper's own verifier input, the per-token tuples (l, m, h, rho) with the
top-K entropy (Sec. 3.1, Eq. 3): :func:`feature_sequence`.

Streaming decode: :class:`StreamState`.
"""

from __future__ import annotations

import ctypes as C

import torch

from . import _abi
from ._abi import (FLAG_BAD_ID, FLAG_BAD_TP, FLAG_NONFINITE, FLAG_OUTSIDE_NUCLEUS,  # noqa: F401
                   ProuterError)

__all__ = ["token_features", "token_features_noalloc", "feature_sequence", "sample_features", "verifier_head", "request_aggregate", "route", "calibrate_threshold",
           "validate_offsets", "StreamState",
           "token_features_workspace", "ProuterError", "FEATURE_FLOATS", "FEATURE_INTS", "PAPER_TOP_K"]

PAPER_TOP_K = 20  # K of the paper's top-K entropy (Sec. 3.1)

FEATURE_FLOATS = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin")
FEATURE_INTS = ("rank", "argmax", "cutoff")
_LINKS = {"identity": 0, "sigmoid": 1}


def _stream_handle() -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t) -> C.c_void_p | None:
    return None if t is None else C.c_void_p(t.data_ptr())


def _dtype_code(logits: torch.Tensor) -> int:
    if logits.dtype == torch.float32:
        return _abi.PR_F32
    if logits.dtype == torch.bfloat16:
        return _abi.PR_BF16
    raise TypeError(f"logits must be float32 or bfloat16, got {logits.dtype}")


def _check_rows(logits, sampled_ids, temperature, top_p):
    if not logits.is_cuda or logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be a 2-D CUDA tensor with unit stride along the vocabulary")
    n = logits.shape[0]
    for name, t, dt in (("sampled_ids", sampled_ids, torch.int32), ("temperature", temperature, torch.float32),
                        ("top_p", top_p, torch.float32)):
        if t is None:
            continue
        if t.dtype != dt or not t.is_cuda or t.dim() != 1 or t.shape[0] != n or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous 1-D {dt} CUDA tensor of length {n}")


def _check_features(f: dict, device, n: int | None, what: str, fields=_abi.FEATURE_FIELDS):
    """Caller-supplied per-token feature tensors: each of `fields` present,
    1-D, contiguous, on `device`, of its dtype, and n long when n is given
    (a tensor on the host would reach a kernel as a host pointer)."""
    for k in fields:
        t = f.get(k)
        dt = torch.float32 if k in FEATURE_FLOATS else torch.int32
        if (t is None or t.dtype != dt or t.device != device or t.dim() != 1 or not t.is_contiguous()
                or (n is not None and t.shape[0] != n)):
            size = "" if n is None else f" of length {n}"
            raise ValueError(f"{what}['{k}'] must be a contiguous 1-D {dt} tensor{size} on {device}")


def _check_workspace(workspace, device):
    if workspace is not None and (workspace.device != device or not workspace.is_contiguous()):
        raise ValueError(f"workspace must be a contiguous tensor on {device}")


def _check_index_tensor(t, name: str, device, n: int | None = None):
    if (t.dtype != torch.int32 or t.device != device or t.dim() != 1 or not t.is_contiguous()
            or (n is not None and t.shape[0] != n)):
        size = "" if n is None else f" [{n}]"
        raise ValueError(f"{name} must be a contiguous int32{size} tensor on {device}")


def _as_row_tensor(x, n, device):
    if isinstance(x, (int, float)):
        return torch.full((n,), float(x), dtype=torch.float32, device=device)
    return x


def _alloc_features(n: int, device) -> dict:
    out = {k: torch.empty(n, dtype=torch.float32, device=device) for k in FEATURE_FLOATS}
    out.update({k: torch.empty(n, dtype=torch.int32, device=device) for k in FEATURE_INTS})
    out["flags"] = torch.empty(n, dtype=torch.int32, device=device)  # uint32 bits
    return out


def _features_struct(f: dict) -> _abi.TokenFeatures:
    return _abi.TokenFeatures(*[f[k].data_ptr() if f.get(k) is not None else None for k in _abi.FEATURE_FIELDS])


def token_features_workspace(logits: torch.Tensor, top_p_on: bool = False) -> int:
    n, V = logits.shape
    return int(_abi.lib().pr_token_features_workspace(_dtype_code(logits), n, V, int(top_p_on)))


def token_features(logits: torch.Tensor, sampled_ids: torch.Tensor, temperature, top_p=None,
                   out: dict | None = None, workspace: torch.Tensor | None = None) -> dict:
    """Per-token features of each logit row (``pr_token_features``).

    ``logits`` [n_rows, V] float32/bfloat16; ``sampled_ids`` int32 [n_rows];
    ``temperature`` float32 [n_rows] or a Python float; ``top_p`` float32
    [n_rows], a Python float or None. Returns a dict of [n_rows] tensors.
    """
    n, V = logits.shape
    temperature = _as_row_tensor(temperature, n, logits.device)
    top_p = None if top_p is None else _as_row_tensor(top_p, n, logits.device)
    _check_rows(logits, sampled_ids, temperature, top_p)
    L = _abi.lib()
    code = _dtype_code(logits)
    if out is None:
        out = _alloc_features(n, logits.device)
    else:
        _check_features(out, logits.device, n, "out")
    _check_workspace(workspace, logits.device)
    need = int(L.pr_token_features_workspace(code, n, V, int(top_p is not None)))
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=logits.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = L.pr_token_features(_ptr(logits), code, n, V, logits.stride(0), _ptr(sampled_ids), _ptr(temperature),
                             _ptr(top_p), C.byref(_features_struct(out)), _ptr(workspace), ws_bytes,
                             _stream_handle())
    _abi.check("pr_token_features", st)
    return out


def token_features_noalloc(logits: torch.Tensor, sampled_ids: torch.Tensor, temperature, top_p=None,
                           out: dict | None = None) -> dict:
    """``pr_token_features_noalloc``: :func:`token_features` with the library's
    static per-GPU scratch instead of a workspace (nothing is allocated by the
    library; pass ``out`` to allocate nothing here either). Calls that overlap
    on one GPU race on that scratch."""
    n, V = logits.shape
    temperature = _as_row_tensor(temperature, n, logits.device)
    top_p = None if top_p is None else _as_row_tensor(top_p, n, logits.device)
    _check_rows(logits, sampled_ids, temperature, top_p)
    if out is None:
        out = _alloc_features(n, logits.device)
    else:
        _check_features(out, logits.device, n, "out")
    st = _abi.lib().pr_token_features_noalloc(_ptr(logits), _dtype_code(logits), n, V, logits.stride(0),
                                              _ptr(sampled_ids), _ptr(temperature), _ptr(top_p),
                                              C.byref(_features_struct(out)), _stream_handle())
    _abi.check("pr_token_features_noalloc", st)
    return out


def feature_sequence(logits: torch.Tensor, sampled_ids: torch.Tensor, temperature, offsets: torch.Tensor,
                     top_p=None, top_k: int = PAPER_TOP_K, features: bool = False, out: torch.Tensor | None = None):
    """The paper's verifier input sequence X (``pr_feature_sequence``).

    Returns X, a float32 [n_rows, 4] tensor of (log-prob of the sampled token,
    max probability, negated top-K entropy, position fraction t / T) per
    row; request i owns rows ``offsets[i]:offsets[i+1]``. With
    ``features=True`` returns ``(X, feats)``, feats being the dict that
    :func:`token_features` returns, computed in the same pass. ``out``: an
    optional float32 [n_rows, 4] CUDA tensor that receives X.
    """
    n, V = logits.shape
    temperature = _as_row_tensor(temperature, n, logits.device)
    top_p = None if top_p is None else _as_row_tensor(top_p, n, logits.device)
    _check_rows(logits, sampled_ids, temperature, top_p)
    if offsets.dtype != torch.int32 or not offsets.is_cuda or offsets.dim() != 1 or not offsets.is_contiguous():
        raise ValueError("offsets must be a contiguous 1-D int32 CUDA tensor")
    if out is not None and (out.dtype != torch.float32 or tuple(out.shape) != (n, 4) or not out.is_contiguous()
                            or out.device != logits.device):
        raise ValueError(f"out must be a contiguous float32 [{n}, 4] tensor on {logits.device}")
    X = torch.empty(n, 4, dtype=torch.float32, device=logits.device) if out is None else out
    feats = _alloc_features(n, logits.device) if features else None
    fs = C.byref(_features_struct(feats)) if feats is not None else None
    st = _abi.lib().pr_feature_sequence(_ptr(logits), _dtype_code(logits), n, V, logits.stride(0),
                                        _ptr(sampled_ids), _ptr(temperature), _ptr(top_p), _ptr(offsets),
                                        offsets.shape[0] - 1, int(top_k), _ptr(X), fs, _stream_handle())
    _abi.check("pr_feature_sequence", st)
    return (X, feats) if features else X


def sample_features(logits: torch.Tensor, temperature, seed: int, offset: int = 0, features: bool = True,
                    offsets: torch.Tensor | None = None, top_k: int = PAPER_TOP_K, ids_out: torch.Tensor | None = None,
                    out: dict | None = None):
    """Fused sample-and-verify (``pr_sample_features``): draws each row's token
    from softmax(logits / T) in the same pass that computes its features.

    Returns ``(ids, feats, X)``: the drawn tokens (int32 [n_rows], -1 where the
    distribution is undefined), the per-token features for them as
    :func:`token_features` returns them (rank written as -1, not available), or None with
    ``features=False``, and the paper's input sequence X for them when
    ``offsets`` is given (else None). The draw is a fixed function of
    (seed, offset, row index, logits, temperature) and of the workgroup size
    the number of rows selects. ``ids_out`` / ``out``: optional preallocated
    outputs (int32 [n_rows]; a features dict as :func:`token_features`
    returns)."""
    n, V = logits.shape
    temperature = _as_row_tensor(temperature, n, logits.device)
    if logits.dim() != 2 or not logits.is_cuda or logits.stride(1) != 1:
        raise ValueError("logits must be a 2-D CUDA tensor with unit column stride")
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("logits must be float32 or bfloat16")
    _check_rows(logits, None, temperature, None)
    if features and out is not None:
        _check_features(out, logits.device, n, "out")
    ids = torch.empty(n, dtype=torch.int32, device=logits.device) if ids_out is None else ids_out
    if ids.dtype != torch.int32 or ids.shape != (n,) or not ids.is_contiguous() or ids.device != logits.device:
        raise ValueError(f"ids_out must be a contiguous int32 [{n}] tensor on {logits.device}")
    feats = (out if out is not None else _alloc_features(n, logits.device)) if features else None
    fs = C.byref(_features_struct(feats)) if feats is not None else None
    X = None
    n_req = 0
    if offsets is not None:
        if offsets.dtype != torch.int32 or not offsets.is_cuda or offsets.dim() != 1 or not offsets.is_contiguous():
            raise ValueError("offsets must be a contiguous 1-D int32 CUDA tensor")
        X = torch.empty(n, 4, dtype=torch.float32, device=logits.device)
        n_req = offsets.shape[0] - 1
    st = _abi.lib().pr_sample_features(_ptr(logits), _dtype_code(logits), n, V, logits.stride(0), _ptr(temperature),
                                       int(seed) & 0xFFFFFFFFFFFFFFFF, int(offset) & 0xFFFFFFFFFFFFFFFF, _ptr(ids),
                                       fs, _ptr(offsets), n_req, int(top_k), _ptr(X), _stream_handle())
    _abi.check("pr_sample_features", st)
    return ids, feats, X


def verifier_head(X: torch.Tensor, offsets: torch.Tensor, weights: torch.Tensor, max_len: int | None = None,
                  workspace: torch.Tensor | None = None) -> torch.Tensor:
    """The paper's shipping confidence per request from its input sequence
    (``pr_verifier_head``). ``X`` float32 [n_rows, 4] (as returned by
    :func:`feature_sequence`), ``offsets`` int32 [n_req + 1], ``weights``
    float32 [67,329] in the documented layout. ``max_len``: at least the
    longest request's length (default: n_rows). Returns float32 [n_req]."""
    if X.dtype != torch.float32 or not X.is_cuda or X.dim() != 2 or X.shape[1] != 4 or not X.is_contiguous():
        raise ValueError("X must be a contiguous float32 [n_rows, 4] CUDA tensor")
    if offsets.dtype != torch.int32 or not offsets.is_cuda or offsets.dim() != 1 or not offsets.is_contiguous():
        raise ValueError("offsets must be a contiguous 1-D int32 CUDA tensor")
    if (weights.dtype != torch.float32 or not weights.is_cuda or weights.numel() != _abi.PR_HEAD_WEIGHTS
            or not weights.is_contiguous()):
        raise ValueError(f"weights must be a contiguous float32 CUDA tensor of {_abi.PR_HEAD_WEIGHTS} entries")
    n = X.shape[0]
    n_req = offsets.shape[0] - 1
    _check_workspace(workspace, X.device)
    L = _abi.lib()
    need = int(L.pr_verifier_head_workspace(n))
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    scores = torch.empty(n_req, dtype=torch.float32, device=X.device)
    st = L.pr_verifier_head(_ptr(X), n, _ptr(offsets), n_req, int(max_len if max_len is not None else max(n, 1)),
                            _ptr(weights), _ptr(scores), _ptr(workspace), ws_bytes, _stream_handle())
    _abi.check("pr_verifier_head", st)
    return scores


def _params(q=0.1, weights=None, bias=0.0, link="identity") -> _abi.AggParams:
    p = _abi.AggParams()
    _abi.lib().pr_agg_params_default(C.byref(p))
    p.q = float(q)
    if weights is not None:
        w = [float(v) for v in torch.as_tensor(weights, dtype=torch.float64).reshape(-1).tolist()]
        if len(w) != 12:
            raise ValueError("weights must have 12 entries (stat-major [mean, min, quant] x 4 features)")
        for i, v in enumerate(w):
            p.w[i] = v
    p.b = float(bias)
    p.link = _LINKS[link]
    return p


def _alloc_agg(n: int, device) -> dict:
    return {"count": torch.empty(n, dtype=torch.int32, device=device),
            "mean": torch.empty(n, 4, dtype=torch.float32, device=device),
            "min": torch.empty(n, 4, dtype=torch.float32, device=device),
            "quant": torch.empty(n, 4, dtype=torch.float32, device=device),
            "score": torch.empty(n, dtype=torch.float32, device=device)}


def _agg_struct(a: dict) -> _abi.RequestAgg:
    return _abi.RequestAgg(*[a[k].data_ptr() if a.get(k) is not None else None for k in _abi.AGG_FIELDS])


def request_aggregate(feats: dict, offsets: torch.Tensor, q: float = 0.1, weights=None, bias: float = 0.0,
                      link: str = "identity") -> dict:
    """Per-request count, mean/min/q-quantile of (logprob, maxprob, -entropy,
    margin) and the summary score (``pr_request_aggregate``)."""
    if offsets.dtype != torch.int32 or not offsets.is_cuda or offsets.dim() != 1 or not offsets.is_contiguous():
        raise ValueError("offsets must be a contiguous 1-D int32 CUDA tensor")
    n_req = offsets.shape[0] - 1
    _check_features(feats, offsets.device, None, "feats", ("logprob", "maxprob", "entropy", "margin"))
    out = _alloc_agg(n_req, offsets.device)
    params = _params(q, weights, bias, link)
    st = _abi.lib().pr_request_aggregate(C.byref(_features_struct(feats)), _ptr(offsets), n_req, C.byref(params),
                                         C.byref(_agg_struct(out)), _stream_handle())
    _abi.check("pr_request_aggregate", st)
    return out


def route(scores: torch.Tensor, threshold: float):
    """Ship iff score >= threshold (``pr_route``). Returns (ship uint8 [n], n_ship int32 [1])."""
    if scores.dtype != torch.float32 or not scores.is_cuda or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous float32 CUDA tensor")
    n = scores.shape[0]
    ship = torch.empty(n, dtype=torch.uint8, device=scores.device)
    n_ship = torch.empty(1, dtype=torch.int32, device=scores.device)
    st = _abi.lib().pr_route(_ptr(scores), n, float(threshold), _ptr(ship), _ptr(n_ship), _stream_handle())
    _abi.check("pr_route", st)
    return ship, n_ship


def calibrate_threshold(scores: torch.Tensor, ship_fraction: float):
    """Threshold tau for a ship fraction on a validation pool of scores
    (``pr_calibrate_threshold``). Returns (tau float32 [1], n_ship int32 [1])."""
    if scores.dtype != torch.float32 or not scores.is_cuda or not scores.is_contiguous() or scores.dim() != 1:
        raise ValueError("scores must be a 1-D contiguous float32 CUDA tensor")
    n = scores.shape[0]
    tau = torch.empty(1, dtype=torch.float32, device=scores.device)
    n_ship = torch.empty(1, dtype=torch.int32, device=scores.device)
    ws_bytes = _abi.lib().pr_calibrate_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=scores.device) if ws_bytes else None
    st = _abi.lib().pr_calibrate_threshold(_ptr(scores), n, float(ship_fraction), _ptr(tau), _ptr(n_ship),
                                          _ptr(ws), ws_bytes, _stream_handle())
    _abi.check("pr_calibrate_threshold", st)
    return tau, n_ship


def validate_offsets(offsets: torch.Tensor, n_rows: int) -> bool:
    """Synchronous check of an offsets array (``pr_validate_offsets``)."""
    if not offsets.is_cuda:
        raise ValueError("offsets must be a CUDA tensor")
    _check_index_tensor(offsets, "offsets", offsets.device)
    st = _abi.lib().pr_validate_offsets(_ptr(offsets), offsets.shape[0] - 1, n_rows, _stream_handle())
    if st == _abi.PR_ERR_INVALID_ARG:
        return False
    _abi.check("pr_validate_offsets", st)
    return True


class StreamState:
    """Device-resident per-request state for streaming decode (``pr_stream_*``).

    ``max_len`` tokens of history per slot give the exact tail quantile;
    ``max_len=0`` keeps P-square markers instead (bounded memory, any length)."""

    def __init__(self, max_slots: int, max_len: int, q: float = 0.1, weights=None, bias: float = 0.0,
                 link: str = "identity"):
        self._h = C.c_void_p()
        params = _params(q, weights, bias, link)
        _abi.check("pr_stream_create", _abi.lib().pr_stream_create(max_slots, max_len, C.byref(params),
                                                                     C.byref(self._h)))
        self.max_slots, self.max_len = max_slots, max_len

    def step(self, logits, slot_ids, sampled_ids, temperature, out: dict | None = None, want_features=False,
             top_p=None):
        n, V = logits.shape
        temperature = _as_row_tensor(temperature, n, logits.device)
        top_p = None if top_p is None else _as_row_tensor(top_p, n, logits.device)
        _check_rows(logits, sampled_ids, temperature, top_p)
        _check_index_tensor(slot_ids, "slot_ids", logits.device, n)
        if out is None and want_features:
            out = _alloc_features(n, logits.device)
        elif out is not None:
            _check_features(out, logits.device, n, "out")
        fs = C.byref(_features_struct(out)) if out is not None else None
        st = _abi.lib().pr_stream_step(self._h, _ptr(logits), _dtype_code(logits), n, V, logits.stride(0),
                                       _ptr(slot_ids), _ptr(sampled_ids), _ptr(temperature), _ptr(top_p), fs,
                                       _stream_handle())
        _abi.check("pr_stream_step", st)
        return out

    def finish(self, slots: torch.Tensor, threshold: float) -> dict:
        if not slots.is_cuda:
            raise ValueError("slots must be a CUDA tensor")
        _check_index_tensor(slots, "slots", slots.device)
        n = slots.shape[0]
        out = _alloc_agg(n, slots.device)
        ship = torch.empty(n, dtype=torch.uint8, device=slots.device)
        st = _abi.lib().pr_stream_finish(self._h, _ptr(slots), n, float(threshold), C.byref(_agg_struct(out)),
                                         _ptr(ship), _stream_handle())
        _abi.check("pr_stream_finish", st)
        out["ship"] = ship
        return out

    def reset(self, slots: torch.Tensor) -> None:
        if not slots.is_cuda:
            raise ValueError("slots must be a CUDA tensor")
        _check_index_tensor(slots, "slots", slots.device)
        _abi.check("pr_stream_reset_slots",
                   _abi.lib().pr_stream_reset_slots(self._h, _ptr(slots), slots.shape[0], _stream_handle()))

    def close(self) -> None:
        if self._h:
            _abi.lib().pr_stream_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
