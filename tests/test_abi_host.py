"""The C-ABI library loads, exports every declared symbol and checks its
host-visible arguments (CPU only: no call here reaches the GPU)."""

import ctypes as C
import os
import re

import pytest

from tests.helpers import ROOT, ensure_built


def declared_symbols():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(pr_[a-z_0-9]+)\s*\(", src))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    lib = ensure_built()
    names = declared_symbols()
    assert "pr_token_features" in names and "pr_request_aggregate" in names and "pr_route" in names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, f"declared but not exported: {missing}"


def test_binding_covers_exports():
    from paper_2608_28726_amd import _abi
    assert sorted(_abi.EXPORTED) == declared_symbols()


def test_status_strings_and_defaults():
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    assert lib.pr_status_string(0) == b"ok"
    assert lib.pr_status_string(1) == b"invalid argument"
    assert lib.pr_status_string(99) == b"unknown status"
    p = _abi.AggParams()
    lib.pr_agg_params_default(C.byref(p))
    assert p.q == 0.1 and p.b == 0.0 and p.link == 0
    assert list(p.w) == [0.0, 1.0] + [0.0] * 10


def test_workspace_sizes():
    lib = ensure_built()
    # Many rows: one workgroup per row, no workspace.
    assert lib.pr_token_features_workspace(1, 16896, 151936, 0) == 0
    # Few long rows: split rows need one 32-byte partial state per workgroup
    # and a 16-byte context record per row.
    ws = lib.pr_token_features_workspace(1, 4, 151936, 0)
    assert ws > 0 and ws % 4 == 0 and (ws // 4 - 16) % 32 == 0 and (ws // 4 - 16) // 32 >= 2
    assert lib.pr_token_features_workspace(0, 0, 100, 0) == 0


@pytest.mark.parametrize("case", ["V<2", "stride<V", "bad dtype", "null logits", "n<0", "null out",
                                  "misaligned"])
def test_invalid_arguments_rejected_on_host(case):
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    feats = _abi.TokenFeatures(*([8] * 10))  # never dereferenced: the call must fail first
    args = dict(logits=C.c_void_p(64), dtype=1, n=4, V=100, stride=100, ids=C.c_void_p(64),
                temps=C.c_void_p(64), out=C.byref(feats))
    if case == "V<2":
        args["V"], args["stride"] = 1, 1
    elif case == "stride<V":
        args["stride"] = 99
    elif case == "bad dtype":
        args["dtype"] = 7
    elif case == "null logits":
        args["logits"] = None
    elif case == "n<0":
        args["n"] = -1
    elif case == "null out":
        args["out"] = None
    elif case == "misaligned":
        args["logits"] = C.c_void_p(65)
    st = lib.pr_token_features(args["logits"], args["dtype"], args["n"], args["V"], args["stride"], args["ids"],
                               args["temps"], None, args["out"], None, 0, None)
    assert st == _abi.PR_ERR_INVALID_ARG


def test_other_entry_points_reject_bad_arguments():
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    assert lib.pr_route(None, 5, 0.5, None, None, None) == _abi.PR_ERR_INVALID_ARG
    assert lib.pr_route(None, -1, 0.5, None, None, None) == _abi.PR_ERR_INVALID_ARG
    agg = _abi.RequestAgg()
    assert lib.pr_request_aggregate(None, None, 3, None, C.byref(agg), None) == _abi.PR_ERR_INVALID_ARG
    assert lib.pr_request_aggregate(None, None, 0, None, C.byref(agg), None) == _abi.PR_OK
    bad = _abi.AggParams()
    lib.pr_agg_params_default(C.byref(bad))
    bad.q = 1.5
    feats = _abi.TokenFeatures(*([8] * 10))
    assert lib.pr_request_aggregate(C.byref(feats), C.c_void_p(64), 3, C.byref(bad), C.byref(agg),
                                    None) == _abi.PR_ERR_INVALID_ARG
    h = C.c_void_p()
    assert lib.pr_stream_create(0, 10, None, C.byref(h)) == _abi.PR_ERR_INVALID_ARG
    assert lib.pr_stream_create(4, -1, None, C.byref(h)) == _abi.PR_ERR_INVALID_ARG  # 0 = bounded memory
    assert lib.pr_stream_step(None, None, 1, 0, 100, 100, None, None, None, None, None, None) == \
        _abi.PR_ERR_INVALID_ARG
    assert lib.pr_stream_finish(None, None, 1, 0.5, None, None, None) == _abi.PR_ERR_INVALID_ARG
    lib.pr_stream_destroy(None)  # ignored
    # zero rows: valid, nothing launched
    feats = _abi.TokenFeatures(*([8] * 10))
    assert lib.pr_token_features(None, 0, 0, 100, 100, None, None, None, C.byref(feats), None, 0, None) == \
        _abi.PR_OK


def test_sample_features_rejects_bad_arguments():
    """pr_sample_features checks everything on the host before any launch."""
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    p = C.c_void_p(256)
    bad = _abi.PR_ERR_INVALID_ARG
    feats = _abi.TokenFeatures(*([8] * 10))
    partial = _abi.TokenFeatures(*([8] * 9 + [0]))
    call = lambda *a: lib.pr_sample_features(*a)
    #          logits dtype n  V   stride T  seed off ids feats          offs n_req k   X     stream
    assert call(p, 7, 4, 100, 100, p, 1, 0, p, C.byref(feats), None, 0, 20, None, None) == bad    # dtype
    assert call(p, _abi.PR_F32, -1, 100, 100, p, 1, 0, p, None, None, 0, 20, None, None) == bad   # n_rows
    assert call(p, _abi.PR_F32, 4, 1, 100, p, 1, 0, p, None, None, 0, 20, None, None) == bad      # vocab < 2
    assert call(p, _abi.PR_F32, 4, 100, 99, p, 1, 0, p, None, None, 0, 20, None, None) == bad     # stride
    assert call(None, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, None, 0, 20, None, None) == bad  # logits
    assert call(p, _abi.PR_F32, 4, 100, 100, None, 1, 0, p, None, None, 0, 20, None, None) == bad  # T
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, None, None, None, 0, 20, None, None) == bad  # ids
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, C.byref(partial), None, 0, 20, None, None) == bad
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, None, 1, 20, p, None) == bad       # X, no offsets
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, p, 1, 0, p, None) == bad           # top_k 0
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, p, 1, 33, p, None) == bad          # top_k > 32
    assert call(p, _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, p, 1, 20, C.c_void_p(260), None) == bad  # X align
    assert call(C.c_void_p(258), _abi.PR_F32, 4, 100, 100, p, 1, 0, p, None, None, 0, 20, None, None) == bad
    assert call(None, _abi.PR_F32, 0, 100, 100, None, 1, 0, None, None, None, 0, 20, None, None) == _abi.PR_OK


def test_topp_vocabulary_limit():
    """The top-p histogram packs a bin's count into 24 bits."""
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    p = C.c_void_p(256)
    V = 1 << 24
    # rejected on the host before any launch
    assert lib.pr_feature_sequence(p, _abi.PR_F32, 4, V, V, p, p, p, p, 1, 20, p, None, None) == \
        _abi.PR_ERR_UNSUPPORTED


def test_calibrate_rejects_bad_arguments():
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    p = C.c_void_p(256)
    bad = _abi.PR_ERR_INVALID_ARG
    assert lib.pr_calibrate_threshold(p, -1, 0.5, p, p, None, 0, None) == bad          # n < 0
    assert lib.pr_calibrate_threshold(None, 4, 0.5, p, p, None, 0, None) == bad        # no scores
    assert lib.pr_calibrate_threshold(p, 4, 0.5, None, p, None, 0, None) == bad        # no tau
    for q in (-0.1, 1.5, float("nan"), float("inf")):
        assert lib.pr_calibrate_threshold(p, 4, q, p, p, None, 0, None) == bad
    assert lib.pr_calibrate_workspace(16384) == 0 and lib.pr_calibrate_workspace(-5) == 0
    need = lib.pr_calibrate_workspace(16385)
    assert need > 0 and lib.pr_calibrate_workspace(1 << 30) == need
    assert lib.pr_calibrate_threshold(p, 16385, 0.5, p, p, None, need, None) == bad    # no workspace
    assert lib.pr_calibrate_threshold(p, 16385, 0.5, p, p, p, need - 4, None) == bad   # too small
    assert lib.pr_calibrate_threshold(p, 16385, 0.5, p, p, C.c_void_p(258), need, None) == bad  # misaligned


@pytest.mark.parametrize("case", ["k=0", "k>max", "null offsets", "no requests", "null X", "misaligned X",
                                  "partial features", "V<2", "n_req<0"])
def test_feature_sequence_rejects_bad_arguments(case):
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    args = dict(logits=C.c_void_p(64), dtype=1, n=4, V=100, stride=100, ids=C.c_void_p(64),
                temps=C.c_void_p(64), offsets=C.c_void_p(64), n_req=2, k=20, X=C.c_void_p(256), feats=None)
    if case == "k=0":
        args["k"] = 0
    elif case == "k>max":
        args["k"] = _abi.PR_MAX_TOP_K + 1
    elif case == "null offsets":
        args["offsets"] = None
    elif case == "no requests":
        args["n_req"] = 0
    elif case == "null X":
        args["X"] = None
    elif case == "misaligned X":
        args["X"] = C.c_void_p(260)
    elif case == "partial features":
        f = _abi.TokenFeatures(*([8] * 9 + [None]))
        args["feats"] = C.byref(f)
    elif case == "V<2":
        args["V"], args["stride"] = 1, 1
    elif case == "n_req<0":
        args["n_req"] = -1
    st = lib.pr_feature_sequence(args["logits"], args["dtype"], args["n"], args["V"], args["stride"], args["ids"],
                                 args["temps"], None, args["offsets"], args["n_req"], args["k"], args["X"],
                                 args["feats"], None)
    assert st == _abi.PR_ERR_INVALID_ARG


def test_feature_sequence_zero_rows_is_valid():
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    assert lib.pr_feature_sequence(None, 1, 0, 100, 100, None, None, None, None, 0, 20, None, None, None) == \
        _abi.PR_OK


def test_verifier_head_rejects_bad_arguments():
    lib = ensure_built()
    from paper_2608_28726_amd import _abi
    p = C.c_void_p(256)
    ws = int(lib.pr_verifier_head_workspace(10))
    # per row: H0, H1, QKV and the attention output (float32), plus the attention's work list
    # (at most 4 items of 2 int32 per row); then the item count and one counter per layer
    assert ws == 10 * ((2 * 64 + 192 + 64) * 4 + 4 * 2 * 4) + (1 + 2) * 4
    assert lib.pr_verifier_head(p, 10, p, 2, 0, p, p, p, ws, None) == _abi.PR_ERR_INVALID_ARG      # max_len < 1
    assert lib.pr_verifier_head(p, -1, p, 2, 8, p, p, p, ws, None) == _abi.PR_ERR_INVALID_ARG      # n_rows < 0
    assert lib.pr_verifier_head(p, 10, None, 2, 8, p, p, p, ws, None) == _abi.PR_ERR_INVALID_ARG   # offsets
    assert lib.pr_verifier_head(p, 10, p, 2, 8, None, p, p, ws, None) == _abi.PR_ERR_INVALID_ARG   # weights
    assert lib.pr_verifier_head(p, 10, p, 2, 8, C.c_void_p(260), p, p, ws, None) == _abi.PR_ERR_INVALID_ARG
    assert lib.pr_verifier_head(p, 10, p, 2, 8, p, p, p, ws - 1, None) == _abi.PR_ERR_INVALID_ARG  # workspace
    assert lib.pr_verifier_head(None, 0, None, 0, 8, None, None, None, 0, None) == _abi.PR_OK       # nothing to do
